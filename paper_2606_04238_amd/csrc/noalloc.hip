// qmlp_forward for callers that cannot allocate device memory (code under
// HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
// the workspace of the block lives in a fixed device array of this library
// instead of a caller buffer.
//
// The array is a file-scope __device__ variable, so every GPU the library
// runs on holds its own copy (at its own address) until the process ends.
// Its address is looked up once per device with hipGetSymbolAddress, with
// that device current, and only that address is handed to kernels and
// copies: in host code the array's name is a host-side stand-in, not a
// device address.
//
// Every call on a GPU shares that GPU's array.  Each call first clears the
// part of it the block uses (the control words and tagged hand-off words of
// the decode kernels must start at zero; a small fill kernel, no memset, so
// the call can be captured in a graph), then runs exactly qmlp_forward on
// it.  Calls that overlap in time on one GPU (two streams, two host
// threads) race on the array.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

#include "qmlp.h"
#include "qmlp_internal.h"

namespace {

constexpr size_t kScratchBytes = (size_t)1 << 20;     // 1 MiB per GPU
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_mu;
void* g_scratch[kMaxDevices];           // device address of `scratch`, per device

// The device address of this GPU's array (current device), looked up on
// the first call on that device.
hipError_t scratch_address(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (!p)
            return hipErrorInvalidSymbol;
        g_scratch[dev] = p;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}

__global__ __launch_bounds__(256) void clear_kernel(uint4* __restrict__ p, long n16) {
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n16; i += (long)gridDim.x * 256)
        p[i] = make_uint4(0u, 0u, 0u, 0u);
}

}  // namespace

extern "C" size_t qmlp_noalloc_scratch_bytes(void) { return kScratchBytes; }

extern "C" qmlp_status qmlp_forward_noalloc(const qmlp_mlp* mlp, const void* x, int M, qmlp_dtype dtype,
                                            void* y, qmlp_stream stream) {
    qmlp_status s = qmlp::forward_check(mlp, x, M, dtype, y);
    if (s != QMLP_OK || M == 0)
        return s;
    if (dtype != QMLP_F16)
        return QMLP_ERR_UNSUPPORTED;
    const size_t need = qmlp_workspace_bytes(mlp, M, dtype);
    if (need == 0 || need > kScratchBytes)
        return QMLP_ERR_WORKSPACE;
    void* ws = nullptr;
    if (scratch_address(&ws) != hipSuccess)
        return QMLP_ERR_HIP;
    hipStream_t st = static_cast<hipStream_t>(stream);
    const long n16 = (long)((need + 15) / 16);
    const int blocks = (int)((n16 + 255) / 256 < 1024 ? (n16 + 255) / 256 : 1024);
    hipLaunchKernelGGL(clear_kernel, dim3(blocks), dim3(256), 0, st, static_cast<uint4*>(ws), n16);
    if (hipGetLastError() != hipSuccess)
        return QMLP_ERR_HIP;
    return qmlp_forward(mlp, x, M, dtype, y, ws, need, stream);
}

// Read-only HBM streaming probe (measurement hook, not part of the MLP).
//
// Decode is bound by loading weights (Sec. 1, Sec. 3.3), so the roofline the
// decode kernels are held to is the HBM read rate.  This kernel reads a
// buffer once with the same 128-bit loads the weight stream uses (the
// non-temporal form, or plain loads for comparison) and does nothing else, so
//   * its duration gives the read rate this GPU actually sustains, and
//   * its byte counters, divided into the known buffer size, calibrate the
//     counters of the decode kernels for loads of the same kind.
// Each thread keeps eight 16-byte loads in flight; the result of every load
// is folded into one XOR word per wave so that no load can be dropped.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qmlp_device.h"
#include "qmlp.h"

namespace qmlp {

namespace {

constexpr int PT = 256;     // threads per workgroup
constexpr int PU = 8;       // loads in flight per thread

template <bool NT>
__device__ __forceinline__ uint4 probe_load(const uint4* p) {
    if constexpr (NT)
        return load_stream(p);
    else
        return *p;
}

template <bool NT>
__global__ __launch_bounds__(PT) void stream_read_kernel(const uint4* __restrict__ p, long n16,
                                                         uint32_t* __restrict__ out) {
    const long stride = (long)gridDim.x * PT;
    long i = (long)blockIdx.x * PT + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (PU - 1) * stride < n16; i += PU * stride) {
        uint4 v[PU];
#pragma unroll
        for (int k = 0; k < PU; ++k) v[k] = probe_load<NT>(p + i + k * stride);
#pragma unroll
        for (int k = 0; k < PU; ++k) acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
    }
    for (; i < n16; i += stride) {
        const uint4 v = probe_load<NT>(p + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
#pragma unroll
    for (int s = 32; s >= 1; s >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, s, 64);
    if ((threadIdx.x & 63) == 0)
        out[(long)blockIdx.x * (PT / 64) + threadIdx.x / 64] = acc;
}

}  // namespace

}  // namespace qmlp

extern "C" qmlp_status qmlp_probe_stream_read(const void* buf, size_t bytes, uint32_t* out, int blocks,
                                              int nontemporal, qmlp_stream stream) {
    using namespace qmlp;
    if (!buf || !out)
        return QMLP_ERR_NULL;
    if (bytes == 0 || bytes % 16 != 0 || blocks < 1 || blocks > 65536)
        return QMLP_ERR_SHAPE;
    if (reinterpret_cast<uintptr_t>(buf) % 16 != 0 || reinterpret_cast<uintptr_t>(out) % 4 != 0)
        return QMLP_ERR_ALIGN;
    const long n16 = (long)(bytes / 16);
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    if (nontemporal)
        hipLaunchKernelGGL(stream_read_kernel<true>, dim3(blocks), dim3(PT), 0, st,
                           reinterpret_cast<const uint4*>(buf), n16, out);
    else
        hipLaunchKernelGGL(stream_read_kernel<false>, dim3(blocks), dim3(PT), 0, st,
                           reinterpret_cast<const uint4*>(buf), n16, out);
    return hipGetLastError() == hipSuccess ? QMLP_OK : QMLP_ERR_HIP;
}

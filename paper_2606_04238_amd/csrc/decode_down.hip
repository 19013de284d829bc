// Stand-alone decode kernel of the 4-bit down projection y = W4down h
// (Sec. 3.3); serves qmlp_down_w4 and the shapes the fused layer kernel does
// not cover.
#include "decode_common.h"
#include "decode_launch.h"

namespace qmlp {

template <int MT, int S, int MAXJ>
__global__ void __launch_bounds__(256)
down_w4_kernel(DownArgs a) {
    extern __shared__ uint4 smem[];
    const int UC = a.uc;
    uint4* hs = smem;
    float2* cx = reinterpret_cast<float2*>(smem + MT * UC * 4);
    const int tid = threadIdx.x, lane = tid & 63;
    DnItem<MT, S, MAXJ> it;
    dn_load(it, a, (blockIdx.x * (blockDim.x >> 6) + (tid >> 6)) * (64 / S), true, lane);
    const int U = a.f / 32;
    for (int u0 = 0; u0 < U; u0 += UC) {
        const int uc = min(UC, U - u0);
        __syncthreads();
        stage_h<MT>(hs, cx, UC, a.h, a.M, a.f, u0, uc, tid, blockDim.x);
        __syncthreads();
        dn_accumulate(it, hs, cx, UC, a.f, u0, uc, lane);
    }
    dn_finish(it, a, lane);
}

#define QMLP_DN_CASE(MT_, S_, J_)                                                         \
    if (mt == MT_ && S == S_ && mj == J_) {                                               \
        auto k = down_w4_kernel<MT_, S_, J_>;                                             \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, 256, lds, st>>>(args);                                                  \
        return hipGetLastError();                                                         \
    }
#define QMLP_DN_S(MT_, S_) QMLP_DN_CASE(MT_, S_, 8) QMLP_DN_CASE(MT_, S_, 16)
#define QMLP_DN_MT(MT_) QMLP_DN_S(MT_, 8) QMLP_DN_S(MT_, 16) QMLP_DN_S(MT_, 32) QMLP_DN_S(MT_, 64)

hipError_t launch_down(DownArgs args, hipStream_t st) {
    const int U = args.f / 32;
    const int S = lanes_down(U);
    const int J = (U + S - 1) / S;
    const int mj = maxj_for(J);
    const int mt = mtile_for(args.M);
    args.uc = units_per_chunk(U, S, DN_UNIT_BYTES, mt);
    const size_t lds = (size_t)mt * args.uc * DN_UNIT_BYTES;
    const int rows_per_block = 4 * (64 / S);
    const dim3 grid((args.d + rows_per_block - 1) / rows_per_block);
    QMLP_DN_MT(1) QMLP_DN_MT(2) QMLP_DN_MT(4) QMLP_DN_MT(8) QMLP_DN_MT(16)
    return hipErrorInvalidValue;
}

}  // namespace qmlp

// Stand-alone decode kernels of the gate/up half: the LoRA-A projection
// t = [A_g; A_u] x and the fused 2-bit gate/up dequant-matvec with the
// LoRA-B term and the SiLU(G) * U epilogue (Sec. 3.1 Eq. (1), Sec. 3.3,
// Sec. 4.2, Sec. 5).  qmlp_forward normally runs the single fused layer
// kernel instead (decode_fused.hip); these serve qmlp_gateup_w2_lora and the
// shapes the fused kernel does not cover.
#include "decode_common.h"
#include "decode_launch.h"

namespace qmlp {

// One wave per row c of [A_g; A_u].
template <int MT>
__global__ void __launch_bounds__(256)
lora_a_kernel(const uint16_t* __restrict__ Ag, const uint16_t* __restrict__ Au,
              const uint16_t* __restrict__ x, int M, int d, int r, float* __restrict__ t) {
    const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
    if (wave >= 2 * r)
        return;
    lora_a_row<MT, (MT <= 4 ? 12 / MT : 1)>(Ag, Au, x, M, d, r, wave, t, threadIdx.x & 63);
}

// Four waves per block, one gate/up item (64/S row pairs) per wave.
template <int MT, int S, int MAXJ>
__global__ void __launch_bounds__(256)
gateup_w2_kernel(GateUpArgs a) {
    extern __shared__ uint4 smem[];
    const int UC = a.uc;
    uint4* xs = smem;
    float2* cx = reinterpret_cast<float2*>(smem + MT * UC * 8);
    const int tid = threadIdx.x, lane = tid & 63;
    GuItem<MT, S, MAXJ> it;
    gu_load(it, a, (blockIdx.x * (blockDim.x >> 6) + (tid >> 6)) * (64 / S), true, lane);
    const int U = a.d / 64;
    for (int u0 = 0; u0 < U; u0 += UC) {
        const int uc = min(UC, U - u0);
        __syncthreads();
        stage_x<MT>(xs, cx, UC, a.x, a.M, a.d, u0, uc, tid, blockDim.x);
        __syncthreads();
        gu_accumulate(it, xs, cx, UC, a.d, u0, uc, lane);
    }
    gu_finish(it, a, a.t, a.h, lane);
}

hipError_t launch_lora_a(const uint16_t* Ag, const uint16_t* Au, const uint16_t* x, int M, int d,
                         int r, float* t, hipStream_t st) {
    const unsigned blocks = (unsigned)((2 * r * 64 + 255) / 256);
    switch (mtile_for(M)) {
    case 1: lora_a_kernel<1><<<blocks, 256, 0, st>>>(Ag, Au, x, M, d, r, t); break;
    case 2: lora_a_kernel<2><<<blocks, 256, 0, st>>>(Ag, Au, x, M, d, r, t); break;
    case 4: lora_a_kernel<4><<<blocks, 256, 0, st>>>(Ag, Au, x, M, d, r, t); break;
    case 8: lora_a_kernel<8><<<blocks, 256, 0, st>>>(Ag, Au, x, M, d, r, t); break;
    default: lora_a_kernel<16><<<blocks, 256, 0, st>>>(Ag, Au, x, M, d, r, t); break;
    }
    return hipGetLastError();
}

#define QMLP_GU_CASE(MT_, S_, J_)                                                         \
    if (mt == MT_ && S == S_ && mj == J_) {                                               \
        auto k = gateup_w2_kernel<MT_, S_, J_>;                                           \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, 256, lds, st>>>(args);                                                  \
        return hipGetLastError();                                                         \
    }
#define QMLP_GU_S(MT_, S_) QMLP_GU_CASE(MT_, S_, 8) QMLP_GU_CASE(MT_, S_, 16)
#define QMLP_GU_MT(MT_) QMLP_GU_S(MT_, 8) QMLP_GU_S(MT_, 16) QMLP_GU_S(MT_, 32) QMLP_GU_S(MT_, 64)

hipError_t launch_gateup(GateUpArgs args, hipStream_t st) {
    const int U = args.d / 64;
    const int S = lanes_gateup(U);
    const int J = (U + S - 1) / S;
    const int mj = maxj_for(J);
    const int mt = mtile_for(args.M);
    args.uc = units_per_chunk(U, S, GU_UNIT_BYTES, mt);
    const size_t lds = (size_t)mt * args.uc * GU_UNIT_BYTES;
    const int rows_per_block = 4 * (64 / S);
    const dim3 grid((args.f + rows_per_block - 1) / rows_per_block);
    QMLP_GU_MT(1) QMLP_GU_MT(2) QMLP_GU_MT(4) QMLP_GU_MT(8) QMLP_GU_MT(16)
    return hipErrorInvalidValue;
}

bool decode_shape_supported(int d, int f) { return decode_shape_supported_impl(d, f); }

}  // namespace qmlp

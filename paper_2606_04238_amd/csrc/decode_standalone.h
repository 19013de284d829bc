// Stand-alone decode kernels as templates over the code width (B), the
// group-32 split (gate/up at 2 or 3 bits) and the block size (NT: 256 threads,
// or 1024 for the down kernel of batches at several tokens).  Each width is instantiated
// in a translation unit of its own (decode_sa_*.hip) so they build in
// parallel; decode_gateup.hip and decode_down.hip dispatch to them.
#pragma once

#include "decode_common.h"
#include "decode_launch.h"

namespace qmlp {

// The descriptor instance l of a batch runs: its own, or on a routed batch
// the routed expert's (read once per workgroup, uniform, clamped to the
// table so an out-of-range id cannot address outside it).
__device__ __forceinline__ int batch_expert(const BatchArgs& b, int l) {
    if (!b.route)
        return l;
    int e = __builtin_amdgcn_readfirstlane(b.route[l]);
    e = e < 0 ? 0 : (e >= b.nexp ? b.nexp - 1 : e);
    return e;
}

// The input of instance l: its own rows, or those of its token group.
__device__ __forceinline__ const uint16_t* batch_x(const BatchArgs& b, int l) {
    return b.x + (long)(b.xdiv > 1 ? l / b.xdiv : l) * b.M * b.d;
}

// Block l of a batch: weights from its descriptor, activations at offset l.
__device__ __forceinline__ GateUpArgs batch_gateup_args(const BatchArgs& b, int l) {
    const StackLayerDesc& w = b.lay[batch_expert(b, l)];
    GateUpArgs a;
    a.cg = w.cg;
    a.mg = w.mg;
    a.cu = w.cu;
    a.mu = w.mu;
    a.x = batch_x(b, l);
    // With rank 0 the item still issues (unused) LoRA-B loads: point them at x.
    a.Bg = b.r > 0 ? w.Bg : a.x;
    a.Bu = b.r > 0 ? w.Bu : a.x;
    a.t = b.t + (long)l * b.M * 2 * b.r;
    a.h = b.h + (long)l * b.M * b.f;
    a.M = b.M;
    a.d = b.d;
    a.f = b.f;
    a.g = b.gg;
    a.r = b.r;
    a.uc = b.uc;
    a.lora_scale = w.lora_scale;
    a.bits = b.bg;
    return a;
}

// NT/64 waves per block, one gate/up item (64/S row pairs) per wave.  B and
// SPLIT as for GuItem: the activation is staged in the layout of the code
// width (eight 16-byte chunks per 64-code unit at 2 bits, four per 32-code
// unit at 4 bits) with one or two (C, X) pairs per unit.
template <int MT, int S, int MAXJ, int B, bool SPLIT, int NT>
__global__ void __launch_bounds__(NT)
gateup_kernel(BatchArgs b) {
    const GateUpArgs a = batch_gateup_args(b, blockIdx.y);
    constexpr int CH = B == 2 ? 8 : B == 3 ? 16 : 4;      // 16-byte chunks per (token, unit)
    extern __shared__ uint4 smem[];
    const int UC = a.uc;
    uint4* xs = smem;
    float2* cx = reinterpret_cast<float2*>(smem + MT * UC * CH);
    const int tid = threadIdx.x, lane = tid & 63;
    GuItem<MT, S, MAXJ, B, SPLIT> it;
    gu_load(it, a, (blockIdx.x * (blockDim.x >> 6) + (tid >> 6)) * (64 / S), true, lane);
    const int U = a.d / codes_per_unit(B);
    for (int u0 = 0; u0 < U; u0 += UC) {
        const int uc = min(UC, U - u0);
        __syncthreads();
        if constexpr (B == 2)
            stage_x<MT, SPLIT>(xs, cx, UC, a.x, a.M, a.d, u0, uc, tid, blockDim.x);
        else if constexpr (B == 3)
            stage_x3<MT, SPLIT>(xs, cx, UC, a.x, a.M, a.d, u0, uc, tid, blockDim.x);
        else
            stage_h<MT>(xs, cx, UC, a.x, a.M, a.d, u0, uc, tid, blockDim.x);
        __syncthreads();
        gu_accumulate(it, xs, cx, UC, a.d, u0, uc, lane);
    }
    gu_finish(it, a, a.t, a.h, lane);
}

#define QMLP_GU_CASE(MT_, S_, J_)                                                         \
    if (mt == MT_ && S == S_ && mj == J_) {                                               \
        auto k = gateup_kernel<MT_, S_, J_, B, SPLIT, NT>;                                \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, NT, lds, st>>>(args);                                                   \
        return hipGetLastError();                                                         \
    }
#define QMLP_GU_S(MT_, S_) QMLP_GU_CASE(MT_, S_, 8) QMLP_GU_CASE(MT_, S_, 16)
#define QMLP_GU_MT(MT_) QMLP_GU_S(MT_, 8) QMLP_GU_S(MT_, 16) QMLP_GU_S(MT_, 32) QMLP_GU_S(MT_, 64)

// S lanes per row (8, 16, 32 or 64, at most 16 units per lane), chosen by
// the dispatcher.
template <int B, bool SPLIT, int NT>
hipError_t launch_gateup_bits(BatchArgs args, int nb, int S, hipStream_t st) {
    const int U = args.d / codes_per_unit(B);
    const int J = (U + S - 1) / S;
    const int mj = maxj_for(J);
    const int mt = mtile_for(args.M);
    const size_t unit_bytes = B == 4 ? DN_UNIT_BYTES : (B == 3 ? 16 : 8) * 16 + 8 * (SPLIT ? 2 : 1);
    args.uc = units_per_chunk(U, S, unit_bytes, mt);
    const size_t lds = (size_t)mt * args.uc * unit_bytes;
    const int rows_per_block = (NT / 64) * (64 / S);
    const dim3 grid((args.f + rows_per_block - 1) / rows_per_block, (unsigned)nb);
    QMLP_GU_MT(1) QMLP_GU_MT(2) QMLP_GU_MT(4) QMLP_GU_MT(8) QMLP_GU_MT(16)
    return hipErrorInvalidValue;
}

// Block l of a batch: weights from its descriptor, h and y at offset l.
__device__ __forceinline__ DownArgs batch_down_args(const BatchArgs& b, int l) {
    DownArgs a;
    const int e = batch_expert(b, l);
    a.cd = b.lay[e].cd;
    a.md = b.lay[e].md;
    a.h = b.h + (long)l * b.M * b.f;
    a.y = b.y + (long)l * b.M * b.d;
    a.M = b.M;
    a.d = b.d;
    a.f = b.f;
    a.g = b.gd;
    a.uc = b.uc;
    a.bits = b.bd;
    return a;
}

// NT/64 waves per block, one down item (64/S rows) per wave.  Every block
// stages all of h, so the rows per block (NT/64 * 64/S) set how many weight
// bytes one staged copy serves.
template <int MT, int S, int MAXJ, int B, int NT>
__global__ void __launch_bounds__(NT)
down_kernel(BatchArgs b) {
    const DownArgs a = batch_down_args(b, blockIdx.y);
    constexpr int CH = B == 2 ? 8 : 4;       // 16-byte chunks of h' per (token, unit)
    extern __shared__ uint4 smem[];
    const int UC = a.uc;
    uint4* hs = smem;
    float2* cx = reinterpret_cast<float2*>(smem + MT * UC * CH);
    const int tid = threadIdx.x, lane = tid & 63;
    DnItem<MT, S, MAXJ, B> it;
    dn_load(it, a, (blockIdx.x * (blockDim.x >> 6) + (tid >> 6)) * (64 / S), true, lane);
    const int U = a.f / codes_per_unit(B);
    for (int u0 = 0; u0 < U; u0 += UC) {
        const int uc = min(UC, U - u0);
        __syncthreads();
        if constexpr (B == 2)
            stage_x<MT>(hs, cx, UC, a.h, a.M, a.f, u0, uc, tid, blockDim.x);
        else
            stage_h<MT>(hs, cx, UC, a.h, a.M, a.f, u0, uc, tid, blockDim.x);
        __syncthreads();
        dn_accumulate(it, hs, cx, UC, a.f, u0, uc, lane);
    }
    dn_finish(it, a, lane);
}

#define QMLP_DN_CASE(MT_, S_, J_)                                                         \
    if (mt == MT_ && S == S_ && mj == J_) {                                               \
        auto k = down_kernel<MT_, S_, J_, B, NT>;                                         \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, NT, lds, st>>>(args);                                                   \
        return hipGetLastError();                                                         \
    }
#define QMLP_DN_S(MT_, S_) QMLP_DN_CASE(MT_, S_, 8) QMLP_DN_CASE(MT_, S_, 16)
#define QMLP_DN_MT(MT_) QMLP_DN_S(MT_, 8) QMLP_DN_S(MT_, 16) QMLP_DN_S(MT_, 32) QMLP_DN_S(MT_, 64)

template <int B, int NT>
hipError_t launch_down_bits(BatchArgs args, int nb, int S, hipStream_t st) {
    const int U = args.f / codes_per_unit(B);
    const int J = (U + S - 1) / S;
    const int mj = maxj_for(J);
    const int mt = mtile_for(args.M);
    const size_t unit_bytes = B == 2 ? GU_UNIT_BYTES : DN_UNIT_BYTES;
    args.uc = units_per_chunk(U, S, unit_bytes, mt);
    const size_t lds = (size_t)mt * args.uc * unit_bytes;
    const int rows_per_block = (NT / 64) * (64 / S);
    const dim3 grid((args.d + rows_per_block - 1) / rows_per_block, (unsigned)nb);
    QMLP_DN_MT(1) QMLP_DN_MT(2) QMLP_DN_MT(4) QMLP_DN_MT(8) QMLP_DN_MT(16)
    return hipErrorInvalidValue;
}

#define QMLP_SA_EXTERN                                                                    \
    extern template hipError_t launch_gateup_bits<2, false, 256>(BatchArgs, int, int, hipStream_t);  \
    extern template hipError_t launch_gateup_bits<2, true, 256>(BatchArgs, int, int, hipStream_t);   \
    extern template hipError_t launch_gateup_bits<4, false, 256>(BatchArgs, int, int, hipStream_t);  \
    extern template hipError_t launch_gateup_bits<3, false, 256>(BatchArgs, int, int, hipStream_t);  \
    extern template hipError_t launch_gateup_bits<3, true, 256>(BatchArgs, int, int, hipStream_t);   \
    extern template hipError_t launch_down_bits<2, 256>(BatchArgs, int, int, hipStream_t);           \
    extern template hipError_t launch_down_bits<2, 1024>(BatchArgs, int, int, hipStream_t);          \
    extern template hipError_t launch_down_bits<4, 256>(BatchArgs, int, int, hipStream_t);           \
    extern template hipError_t launch_down_bits<4, 1024>(BatchArgs, int, int, hipStream_t);

}  // namespace qmlp

// Stand-alone decode kernels as templates over the code width (B), the
// group-32 split (gate/up at 2 or 3 bits) and the block size (NT: 256 threads,
// or 1024 for the down kernel of batches at several tokens).  Each width is instantiated
// in a translation unit of its own (decode_sa_*.hip) so they build in
// parallel; decode_gateup.hip and decode_down.hip dispatch to them.
#pragma once

#include <type_traits>

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
// unit at 4 bits) with one or two (C, X) pairs per unit.  NXW > 0 (one
// token, the activation in one staging pass of NXW words per thread): the
// activation loads go out before the weights, so the staging converts while
// the weight stream is in flight (loads retire in order).
template <int MT, int S, int MAXJ, int B, bool SPLIT, int NT, int NXW = 0>
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
    const int row0 = (blockIdx.x * (NT >> 6) + (tid >> 6)) * (64 / S);
    const int U = a.d / codes_per_unit(B);
    if constexpr (NXW > 0) {
        static_assert(MT == 1, "one staging pass at one token");
        using HW = typename std::conditional<B == 4, uint4, XWord>::type;
        HW xw[NXW];
#pragma unroll
        for (int k = 0; k < NXW; ++k) {
            if constexpr (B == 4)
                xw[k] = stage_h_load<1>(a.x, 1, a.d, 0, U, tid + NT * k);
            else
                xw[k] = stage_x_load<1>(a.x, 1, a.d, 0, U, tid + NT * k);
        }
        __builtin_amdgcn_sched_barrier(0);          // keep the activation loads ahead of the weights
        gu_load(it, a, row0, true, lane);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < NXW; ++k) {
            if constexpr (B == 2)
                stage_x_store<1, SPLIT>(xs, cx, U, U, 1, tid + NT * k, xw[k]);
            else if constexpr (B == 3)
                stage_x3_store<1, SPLIT>(xs, cx, U, U, 1, tid + NT * k, xw[k]);
            else
                stage_h_store<1>(xs, cx, U, U, 1, tid + NT * k, xw[k]);
        }
        __syncthreads();
        gu_accumulate(it, xs, cx, U, a.d, 0, U, lane);
        gu_finish(it, a, a.t, a.h, lane);
        return;
    }
    gu_load(it, a, row0, true, lane);
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

// ---- gate/up over routed instances at one token, with the LoRA-A
// projection in the same launch.  With rank r > 0, workgroup column x < LB
// of instance l (LB = 2r/4 rounded up) computes four rows c of
// t_l = [A_g; A_u] x_l, one per wave, and publishes each as a tagged word
// (fp32 bits | tag << 32, tag = the call counter plus one, never 0) with a
// device-coherent store.  The other columns run the gate/up item: with
// NXW > 0 (the activation fits one staging pass at NXW words per thread)
// the activation loads go out BEFORE the weights, so its staging converts
// while the weight stream is still in flight (loads retire in order);
// otherwise the chunk loop of gateup_kernel.  After the staging barrier the
// block's first 2r threads issue device-coherent loads of t_l, and before
// the epilogue they re-read any word that does not yet show this call's tag
// (bounded: after kTagSpinLimit polls the word is taken as it is and error
// bit 1 is set).  The LoRA-A columns of an instance precede its gate/up
// columns in dispatch order, so every wait is on a workgroup that is already
// resident.
constexpr unsigned kTagSpinLimit = 1u << 18;

template <int S, int MAXJ, int B, bool SPLIT, int NXW>
__global__ void __launch_bounds__(256)
gateup_routed_kernel(BatchArgs b, unsigned long long* t64, unsigned* ctl, int LB) {
    const int l = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const unsigned epoch = __hip_atomic_load(ctl + kMoeCtlEpoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned tag = epoch % 0xFFFFFFFFu + 1u;
    unsigned long long* tl = t64 + (long)l * 2 * b.r;
    if ((int)blockIdx.x < LB) {
        const int c = blockIdx.x * 4 + wave;
        if (c < 2 * b.r) {
            const StackLayerDesc& w = b.lay[batch_expert(b, l)];
            const uint16_t* arow = c < b.r ? w.Ag + (long)c * b.d : w.Au + (long)(c - b.r) * b.d;
            const float v = lora_a_dot<12>(arow, batch_x(b, l), b.d, lane);
            if (lane == 0)
                __hip_atomic_store(tl + c, (unsigned long long)__float_as_uint(v) | ((unsigned long long)tag << 32),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        return;
    }
    GateUpArgs a = batch_gateup_args(b, l);
    constexpr int CH = B == 2 ? 8 : B == 3 ? 16 : 4;
    extern __shared__ uint4 smem[];
    __shared__ float ts[64];
    const int UC = a.uc;
    uint4* xs = smem;
    float2* cx = reinterpret_cast<float2*>(smem + UC * CH);
    GuItem<1, S, MAXJ, B, SPLIT, false> it;
    const int row0 = ((blockIdx.x - LB) * 4 + wave) * (64 / S);
    const int U = a.d / codes_per_unit(B);
    const bool poll = tid < 2 * a.r;
    unsigned long long tv = 0;
    if constexpr (NXW > 0) {
        // one pass (UC = U): words past 4U load word 0 and are dropped
        using HW = typename std::conditional<B == 4, uint4, XWord>::type;
        HW xw[NXW];
#pragma unroll
        for (int k = 0; k < NXW; ++k) {
            if constexpr (B == 4)
                xw[k] = stage_h_load<1>(a.x, 1, a.d, 0, U, tid + 256 * k);
            else
                xw[k] = stage_x_load<1>(a.x, 1, a.d, 0, U, tid + 256 * k);
        }
        __builtin_amdgcn_sched_barrier(0);          // keep the activation loads ahead of the weights
        gu_load(it, a, row0, true, lane);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int k = 0; k < NXW; ++k) {
            if constexpr (B == 2)
                stage_x_store<1, SPLIT>(xs, cx, U, U, 1, tid + 256 * k, xw[k]);
            else if constexpr (B == 3)
                stage_x3_store<1, SPLIT>(xs, cx, U, U, 1, tid + 256 * k, xw[k]);
            else
                stage_h_store<1>(xs, cx, U, U, 1, tid + 256 * k, xw[k]);
        }
        __syncthreads();
        if (poll)
            tv = __hip_atomic_load(tl + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        gu_accumulate(it, xs, cx, U, a.d, 0, U, lane);
    } else {
        gu_load(it, a, row0, true, lane);
        for (int u0 = 0; u0 < U; u0 += UC) {
            const int uc = min(UC, U - u0);
            __syncthreads();
            if constexpr (B == 2)
                stage_x<1, SPLIT>(xs, cx, UC, a.x, 1, a.d, u0, uc, tid, 256);
            else if constexpr (B == 3)
                stage_x3<1, SPLIT>(xs, cx, UC, a.x, 1, a.d, u0, uc, tid, 256);
            else
                stage_h<1>(xs, cx, UC, a.x, 1, a.d, u0, uc, tid, 256);
            __syncthreads();
            if (u0 == 0 && poll)
                tv = __hip_atomic_load(tl + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            gu_accumulate(it, xs, cx, UC, a.d, u0, uc, lane);
        }
    }
    if (poll) {
        for (unsigned n = 0; (unsigned)(tv >> 32) != tag && n < kTagSpinLimit; ++n) {
            __builtin_amdgcn_s_sleep(2);
            tv = __hip_atomic_load(tl + tid, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if ((unsigned)(tv >> 32) != tag)
            __hip_atomic_fetch_or(ctl + kMoeCtlErr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ts[tid] = __uint_as_float((uint32_t)tv);
    }
    __syncthreads();
    gu_finish(it, a, ts, a.h, lane);
}

#define QMLP_GUR_CASE(S_, J_, X_)                                                         \
    if (S == S_ && mj == J_ && nxw == X_) {                                               \
        auto k = gateup_routed_kernel<S_, J_, B, SPLIT, X_>;                              \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, 256, lds, st>>>(args, t64, ctl, LB);                                    \
        return hipGetLastError();                                                         \
    }
#define QMLP_GUR_S(S_) QMLP_GUR_CASE(S_, 8, 0) QMLP_GUR_CASE(S_, 16, 0) QMLP_GUR_CASE(S_, 8, 1) \
    QMLP_GUR_CASE(S_, 16, 1) QMLP_GUR_CASE(S_, 8, 2) QMLP_GUR_CASE(S_, 16, 2)

// Routed instances at one token, rank 0 or 8..32: LB LoRA-A columns (none
// at rank 0), then the gate/up columns of launch_gateup_bits's shape at S
// lanes per row; the activation is loaded ahead of the weights when one
// staging pass of at most two words per thread holds it.
template <int B, bool SPLIT>
hipError_t launch_gateup_routed_bits(BatchArgs args, int nb, int S, unsigned long long* t64, unsigned* ctl,
                                     hipStream_t st) {
    if (args.M != 1 || args.r < 0 || 2 * args.r > 64 || !t64 || !ctl)
        return hipErrorInvalidValue;
    const int U = args.d / codes_per_unit(B);
    const int J = (U + S - 1) / S;
    const int mj = maxj_for(J);
    const size_t unit_bytes = B == 4 ? DN_UNIT_BYTES : (B == 3 ? 16 : 8) * 16 + 8 * (SPLIT ? 2 : 1);
    args.uc = units_per_chunk(U, S, unit_bytes, 1);
    const int nxw = args.uc >= U && 4 * U <= 256 * 2 ? (4 * U + 255) / 256 : 0;
    const size_t lds = (size_t)args.uc * unit_bytes;
    const int LB = (2 * args.r + 3) / 4;
    const int rows_per_block = 4 * (64 / S);
    const dim3 grid((unsigned)(LB + (args.f + rows_per_block - 1) / rows_per_block), (unsigned)nb);
    QMLP_GUR_S(8) QMLP_GUR_S(16) QMLP_GUR_S(32) QMLP_GUR_S(64)
    return hipErrorInvalidValue;
}

#define QMLP_GU_CASE(MT_, S_, J_)                                                         \
    if (mt == MT_ && S == S_ && mj == J_ && (MT_ > 1 || nxw == 0)) {                      \
        auto k = gateup_kernel<MT_, S_, J_, B, SPLIT, NT>;                                \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, NT, lds, st>>>(args);                                                   \
        return hipGetLastError();                                                         \
    }
#define QMLP_GU_X(S_, J_, X_)                                                             \
    if (mt == 1 && S == S_ && mj == J_ && nxw == X_) {                                    \
        auto k = gateup_kernel<1, S_, J_, B, SPLIT, NT, X_>;                              \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, NT, lds, st>>>(args);                                                   \
        return hipGetLastError();                                                         \
    }
#define QMLP_GU_S(MT_, S_) QMLP_GU_CASE(MT_, S_, 8) QMLP_GU_CASE(MT_, S_, 16)
#define QMLP_GU_MT(MT_) QMLP_GU_S(MT_, 8) QMLP_GU_S(MT_, 16) QMLP_GU_S(MT_, 32) QMLP_GU_S(MT_, 64)
#define QMLP_GU_XS(S_) QMLP_GU_X(S_, 8, 1) QMLP_GU_X(S_, 16, 1) QMLP_GU_X(S_, 8, 2) QMLP_GU_X(S_, 16, 2)

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
    // one token whose activation fits one staging pass of at most two words
    // per thread: the activation-first form
    const int nxw = mt == 1 && args.uc >= U && 4 * U <= 2 * NT ? (4 * U + NT - 1) / NT : 0;
    QMLP_GU_XS(8) QMLP_GU_XS(16) QMLP_GU_XS(32) QMLP_GU_XS(64)
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

// ---- software-pipelined down kernel: batches at one token.
// Each wave owns NI consecutive items of 64/S rows; the loads of item k+1
// are issued before item k is computed (two register sets, straight-line
// code), so a wave keeps a load stream in flight through its arithmetic
// instead of alternating "all loads, then all compute".  h is staged once
// per workgroup for 4 * NI items.  JJ = units per lane, exact (every slot
// loads, from a clamped address when past the row).
constexpr int kPipeItems = 4;
constexpr int kPipeMaxUnits = 6;                     // JJ: units per lane
constexpr int kPipeStageWords = 6;                   // staging words per thread: U <= 384

template <int JJ>
struct PipeItem {
    uint4 q[JJ];
    uint32_t m[JJ];
};

template <int S, int JJ, int B>
__device__ __forceinline__ void pipe_load(PipeItem<JJ>& it, const DownArgs& a, int U, int row,
                                          int lane) {
    const int s = lane % S;
    const int upg = a.g / codes_per_unit(B);
    const long rowc = row < a.d ? row : 0;
    const uint4* cd = reinterpret_cast<const uint4*>(a.cd) + rowc * U;
    const uint32_t* md = a.md + rowc * (a.f / a.g);
#pragma unroll
    for (int i = 0; i < JJ; ++i) {
        const int u = s + S * i;
        const int uu = u < U ? u : 0;
        it.q[i] = load_stream(cd + uu);
        it.m[i] = load_stream(md + uu / upg);
    }
}

// s (sum q h' - C - z X) over the lane's units of one row (M = 1, h staged
// whole: unit ul at chunk offset ul).
template <int S, int JJ, int B>
__device__ __forceinline__ float pipe_dot(PipeItem<JJ>& it, const uint4* hs, const float2* cx,
                                          int U, int lane) {
    const uint32_t mv = 0x64006400u;
    const int s = lane % S;
    float y = 0.0f;
#pragma unroll
    for (int i = 0; i < JJ; ++i) {
        const int ul = s + S * i;
        if (ul < U) {
            uint32_t wv[4] = {it.q[i].x, it.q[i].y, it.q[i].z, it.q[i].w};
            uint32_t mi = it.m[i];
#pragma unroll
            for (int w = 0; w < 4; ++w) pin(wv[w]);
            pin(mi);
            float acc = 0.0f;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                if constexpr (B == 4) {
                    uint32_t e[4];
                    extract_w4(wv[w], e, mv);
                    const uint4 p = hs[ul * 4 + (w ^ ((ul >> 1) & 3))];
                    acc = dot2(e[0], p.x, acc);
                    acc = dot2(e[1], p.y, acc);
                    acc = dot2(e[2], p.z, acc);
                    acc = dot2(e[3], p.w, acc);
                } else {
                    uint32_t e[8];
                    extract_w2(wv[w], e, mv);
                    const uint4 p0 = hs[ul * 8 + ((2 * w) ^ (ul & 7))];
                    const uint4 p1 = hs[ul * 8 + ((2 * w + 1) ^ (ul & 7))];
                    const uint32_t hp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
                    for (int p = 0; p < 8; ++p) acc = dot2(e[p], hp[p], acc);
                }
            }
            const float2 k = cx[ul];
            y += h2f(mi & 0xFFFFu) * (acc - k.x - h2f(mi >> 16) * k.y);
        }
    }
    return y;
}

template <int S, int JJ, int B, int NI>
__global__ void __launch_bounds__(256)
down_pipe_kernel(BatchArgs b) {
    const DownArgs a = batch_down_args(b, blockIdx.y);
    constexpr int CH = B == 2 ? 8 : 4;
    constexpr int RPI = 64 / S;                      // rows per item
    extern __shared__ uint4 smem[];
    const int U = a.f / codes_per_unit(B);
    uint4* hs = smem;
    float2* cx = reinterpret_cast<float2*>(smem + U * CH);
    const int tid = threadIdx.x, lane = tid & 63;
    const int row0 = (blockIdx.x * 4 + (tid >> 6)) * NI * RPI + lane / S;
    // h is loaded BEFORE the first item's weights: loads retire in order, so
    // the staging can convert it while the weight stream is still in flight
    // (4 U staging words, at most kPipeStageWords per thread; the loads of
    // words past the end read word 0 and are dropped by the store).
    using HW = typename std::conditional<B == 2, XWord, uint4>::type;
    HW hv[kPipeStageWords];
#pragma unroll
    for (int j = 0; j < kPipeStageWords; ++j) {
        if constexpr (B == 2)
            hv[j] = stage_x_load<1>(a.h, 1, a.f, 0, U, tid + 256 * j);
        else
            hv[j] = stage_h_load<1>(a.h, 1, a.f, 0, U, tid + 256 * j);
    }
    __builtin_amdgcn_sched_barrier(0);              // keep the h loads ahead of the weights
    PipeItem<JJ> buf[2];
    pipe_load<S, JJ, B>(buf[0], a, U, row0, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < kPipeStageWords; ++j) {
        if constexpr (B == 2)
            stage_x_store<1>(hs, cx, U, U, 1, tid + 256 * j, hv[j]);
        else
            stage_h_store<1>(hs, cx, U, U, 1, tid + 256 * j, hv[j]);
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NI; ++k) {
        if (k + 1 < NI)
            pipe_load<S, JJ, B>(buf[(k + 1) & 1], a, U, row0 + (k + 1) * RPI, lane);
        const float v = group_sum<S>(pipe_dot<S, JJ, B>(buf[k & 1], hs, cx, U, lane));
        const int row = row0 + k * RPI;
        if (lane % S == 0 && row < a.d)
            a.y[row] = (uint16_t)f2h(v);
    }
}

// ---- the pipelined down kernel over routed instances with the combine of
// the MoE layer folded in (k <= 4 instances per token, one token per
// workgroup row of the grid).  The workgroup's waves are split into
// G = 4 / k row groups of k waves; wave j of a group runs instance (token,
// slot j) over the group's NI items, so all k instances of an output row are
// computed in one workgroup.  The workgroup stages the h of its k instances
// (k * 4U staging words, at most kPipeStageWords per thread), each wave puts
// its fp32 rows into LDS, and after one barrier the sum over the slots in
// order, w[m][j] y_j from j = 0, is rounded once to binary16 into y[m].
// Waves past G * k (k = 3) only stage.
template <int S, int JJ, int B, int NI>
__global__ void __launch_bounds__(256)
down_pipe_combine_kernel(BatchArgs b, const float* __restrict__ w, uint16_t* __restrict__ y,
                         unsigned* ctl) {
    constexpr int CH = B == 2 ? 8 : 4;
    constexpr int RPI = 64 / S;                      // rows per item
    constexpr int RPW = NI * RPI;                    // rows per wave
    const int k = b.xdiv, G = 4 / k, m = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int j = wave % k, grp = wave / k;
    const bool active = grp < G;
    if (ctl && tid == 0 && blockIdx.x == 0 && blockIdx.y == 0)
        advance_call_counter(ctl + kMoeCtlEpoch);
    const DownArgs a = batch_down_args(b, m * k + (active ? j : 0));
    extern __shared__ uint4 smem[];
    __shared__ float part[4][4 * RPW];
    const int U = a.f / codes_per_unit(B);
    uint4* hs = smem;
    float2* cx = reinterpret_cast<float2*>(smem + k * U * CH);
    const int rbase = blockIdx.x * G * RPW;          // first output row of the workgroup
    const int row0 = rbase + (active ? grp : 0) * RPW + lane / S;
    // staging word t: instance slot t / 4U, word t % 4U of its h (a word past
    // the k instances is given an index past the end: it loads word 0 and
    // its store is dropped)
    const uint16_t* hb = b.h + (long)m * k * a.f;
    using HW = typename std::conditional<B == 2, XWord, uint4>::type;
    HW hv[kPipeStageWords];
#pragma unroll
    for (int i = 0; i < kPipeStageWords; ++i) {
        const int t = tid + 256 * i, sl = min(t / (4 * U), k - 1), wl = t - sl * 4 * U;
        if constexpr (B == 2)
            hv[i] = stage_x_load<1>(hb + (long)sl * a.f, 1, a.f, 0, U, wl);
        else
            hv[i] = stage_h_load<1>(hb + (long)sl * a.f, 1, a.f, 0, U, wl);
    }
    __builtin_amdgcn_sched_barrier(0);              // keep the h loads ahead of the weights
    PipeItem<JJ> buf[2];
    pipe_load<S, JJ, B>(buf[0], a, U, row0, lane);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kPipeStageWords; ++i) {
        const int t = tid + 256 * i, sl = min(t / (4 * U), k - 1), wl = t - sl * 4 * U;
        if constexpr (B == 2)
            stage_x_store<1>(hs + sl * U * CH, cx + sl * U, U, U, 1, wl, hv[i]);
        else
            stage_h_store<1>(hs + sl * U * CH, cx + sl * U, U, U, 1, wl, hv[i]);
    }
    __syncthreads();
    if (active) {
        const uint4* hj = hs + j * U * CH;
        const float2* cj = cx + j * U;
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            if (it + 1 < NI)
                pipe_load<S, JJ, B>(buf[(it + 1) & 1], a, U, row0 + (it + 1) * RPI, lane);
            const float v = group_sum<S>(pipe_dot<S, JJ, B>(buf[it & 1], hj, cj, U, lane));
            if (lane % S == 0)
                part[j][grp * RPW + it * RPI + lane / S] = v;
        }
    }
    __syncthreads();
    if (tid < G * RPW && rbase + tid < a.d) {
        float acc = 0.0f;
        for (int s = 0; s < k; ++s)
            acc += w[m * k + s] * part[s][tid];
        y[(long)m * a.d + rbase + tid] = (uint16_t)f2h(acc);
    }
}


// The pipelined kernel serves M = 1 launches whose whole h fits the LDS
// budget; S = the fewest lanes per row with at most kPipeMaxUnits units each.
inline int pipe_lanes(int U) {
    if (4 * U > 256 * kPipeStageWords)
        return 0;
    for (int S = 8; S <= 64; S *= 2)
        if ((U + S - 1) / S <= kPipeMaxUnits) return S;
    return 0;
}

// Compute units of the current device (an immutable property, cached per
// device); 0 without one.
inline int device_cu_count() {
    static int cache[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
        return 0;
    if (cache[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        cache[dev] = n;
    }
    return cache[dev];
}

// Lanes per row of a routed launch (a few expert instances of one token):
// the launch's usual choice doubled (more, shorter rows per workgroup) while
// it has fewer than two workgroups per compute unit, up to 64 lanes and one
// 16-byte unit per lane.  blocks(S) = the launch's workgroups at S lanes.
template <typename Blocks>
inline int routed_lanes(int S, int U, int cus, Blocks blocks) {
    while (S < 64 && 2 * S <= U && blocks(S) < 2L * cus)
        S *= 2;
    return S;
}
// Gate/up over nb instances of f rows (256-thread workgroups, 256 / S rows each).
inline int routed_gateup_lanes(int U, int f, int nb, int bits, int cus) {
    return routed_lanes(lanes_for(U, bits), U, cus,
                        [&](int s) { return (long)((f + 256 / s - 1) / (256 / s)) * nb; });
}
// The pipelined down kernel over nb instances of d rows (0: it does not take U).
inline int routed_pipe_lanes(int U, int d, int nb, int cus) {
    const int S = pipe_lanes(U);
    if (S == 0)
        return 0;
    return routed_lanes(S, U, cus, [&](int s) {
        const int rpb = 4 * kPipeItems * (64 / s);
        return (long)((d + rpb - 1) / rpb) * nb;
    });
}

#define QMLP_PIPE_CASE(S_, J_)                                                            \
    if (S == S_ && JJ == J_) {                                                            \
        auto k = down_pipe_kernel<S_, J_, B, kPipeItems>;                                 \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, 256, lds, st>>>(args);                                                  \
        return hipGetLastError();                                                         \
    }
#define QMLP_PIPE_S(S_) QMLP_PIPE_CASE(S_, 1) QMLP_PIPE_CASE(S_, 2) QMLP_PIPE_CASE(S_, 3) \
    QMLP_PIPE_CASE(S_, 4) QMLP_PIPE_CASE(S_, 5) QMLP_PIPE_CASE(S_, 6)

template <int B>
hipError_t launch_down_pipe(const BatchArgs& args, int nb, hipStream_t st) {
    const int U = args.f / codes_per_unit(B);
    const int S = args.route ? routed_pipe_lanes(U, args.d, nb, device_cu_count()) : pipe_lanes(U);
    const int JJ = S ? (U + S - 1) / S : 0;
    const size_t lds = (size_t)U * (B == 2 ? GU_UNIT_BYTES : DN_UNIT_BYTES);
    const int rows_per_block = 4 * kPipeItems * (64 / (S ? S : 64));
    const dim3 grid((args.d + rows_per_block - 1) / rows_per_block, (unsigned)nb);
    QMLP_PIPE_S(8) QMLP_PIPE_S(16) QMLP_PIPE_S(32) QMLP_PIPE_S(64)
    return hipErrorInvalidValue;
}

#define QMLP_PIPE_CMB_CASE(S_, J_)                                                        \
    if (S == S_ && JJ == J_) {                                                            \
        auto kf = down_pipe_combine_kernel<S_, J_, B, kPipeItems>;                        \
        hipError_t e = set_lds(kf, lds);                                                  \
        if (e != hipSuccess) return e;                                                    \
        kf<<<grid, 256, lds, st>>>(args, w, y, ctl);                                      \
        return hipGetLastError();                                                         \
    }
#define QMLP_PIPE_CMB_S(S_) QMLP_PIPE_CMB_CASE(S_, 1) QMLP_PIPE_CMB_CASE(S_, 2)             \
    QMLP_PIPE_CMB_CASE(S_, 3) QMLP_PIPE_CMB_CASE(S_, 4) QMLP_PIPE_CMB_CASE(S_, 5)         \
    QMLP_PIPE_CMB_CASE(S_, 6)

// Lanes per row of down_pipe_combine_kernel: the fewest with at most
// kCombineUnits units per lane.  A workgroup stages the h of all k
// instances of its token, so fewer, longer rows per lane spread that staging
// over more rows: at GPT-OSS-20B-class experts (f = 2880, top-4) 3 units per
// lane measured fastest at both down widths (4 bits: 32 lanes, 2 bits: 16),
// ahead of 2 (20.2 against 21.2 us per W4/W2-GateUp layer; 18.8 against
// 20.1 at uniform W2) and 6.
constexpr int kCombineUnits = 3;
inline int combine_lanes(int U) {
    for (int S = 8; S <= 64; S *= 2)
        if ((U + S - 1) / S <= kCombineUnits) return S;
    return pipe_lanes(U);
}

// Whether down_pipe_combine_kernel takes a routed batch of ntok * k
// instances at one token each: k <= 4, h of the k instances within the
// staging words and the LDS budget, and the lanes per row of the routed
// pipelined launch.
inline bool down_combine_fits_shape(int d, int f, int k, int bits) {
    const int U = f / codes_per_unit(bits);
    return k >= 1 && k <= 4 && d >= 1 && pipe_lanes(U) != 0 && k * 4 * U <= 256 * kPipeStageWords &&
           (size_t)k * U * (bits == 2 ? GU_UNIT_BYTES : DN_UNIT_BYTES) <= (size_t)kLdsBudget;
}

// y [ntok][d] = sum_j w[m][j] * down(instance m k + j): args is the routed
// batch (M = 1, xdiv = k), nb = ntok * k; the caller checks
// down_combine_fits_shape first.
template <int B>
hipError_t launch_down_pipe_combine(const BatchArgs& args, int nb, const float* w, uint16_t* y,
                                    unsigned* ctl, hipStream_t st) {
    const int k = args.xdiv;
    const int U = args.f / codes_per_unit(B);
    const int S = combine_lanes(U);
    const int JJ = S ? (U + S - 1) / S : 0;
    if (!S || k < 1 || k > 4 || nb % k != 0)
        return hipErrorInvalidValue;
    const size_t lds = (size_t)k * U * (B == 2 ? GU_UNIT_BYTES : DN_UNIT_BYTES);
    const int rows_per_block = (4 / k) * kPipeItems * (64 / S);
    const dim3 grid((args.d + rows_per_block - 1) / rows_per_block, (unsigned)(nb / k));
    QMLP_PIPE_CMB_S(8) QMLP_PIPE_CMB_S(16) QMLP_PIPE_CMB_S(32) QMLP_PIPE_CMB_S(64)
    return hipErrorInvalidValue;
}

// Batches, and single launches with rows enough to fill the chip in
// workgroups of 4 * kPipeItems items (an LM head).
constexpr int kPipeSingleMinRows = 16384;

inline bool down_pipe_fits_shape(int d, int f, int M, int nb, int bits) {
    const int U = f / codes_per_unit(bits);
    return (nb > 1 || d >= kPipeSingleMinRows) && M == 1 && pipe_lanes(U) != 0 &&
           (size_t)U * (bits == 2 ? GU_UNIT_BYTES : DN_UNIT_BYTES) <= (size_t)kLdsBudget;
}
template <int B>
bool down_pipe_fits(const BatchArgs& args, int nb) {
    return down_pipe_fits_shape(args.d, args.f, args.M, nb, B);
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
    if (NT == 256 && down_pipe_fits<B>(args, nb))
        return launch_down_pipe<B>(args, nb, st);
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
    extern template hipError_t launch_gateup_routed_bits<2, false>(BatchArgs, int, int, unsigned long long*, \
                                                                 unsigned*, hipStream_t);            \
    extern template hipError_t launch_gateup_routed_bits<2, true>(BatchArgs, int, int, unsigned long long*,  \
                                                                unsigned*, hipStream_t);             \
    extern template hipError_t launch_gateup_routed_bits<3, false>(BatchArgs, int, int, unsigned long long*, \
                                                                 unsigned*, hipStream_t);            \
    extern template hipError_t launch_gateup_routed_bits<3, true>(BatchArgs, int, int, unsigned long long*,  \
                                                                unsigned*, hipStream_t);             \
    extern template hipError_t launch_gateup_routed_bits<4, false>(BatchArgs, int, int, unsigned long long*, \
                                                                 unsigned*, hipStream_t);            \
    extern template hipError_t launch_down_bits<2, 256>(BatchArgs, int, int, hipStream_t);           \
    extern template hipError_t launch_down_bits<2, 1024>(BatchArgs, int, int, hipStream_t);          \
    extern template hipError_t launch_down_bits<4, 256>(BatchArgs, int, int, hipStream_t);           \
    extern template hipError_t launch_down_bits<4, 1024>(BatchArgs, int, int, hipStream_t);

}  // namespace qmlp

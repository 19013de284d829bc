// Building blocks of the decode kernels (1 <= M <= 16, binary16), gfx950.
//
// The block (arXiv 2606.04238):
//   G = W2gate x + s_L B_g (A_g x),  U = W2up x + s_L B_u (A_u x)   (Sec. 3.1 Eq. (1), Sec. 4.2)
//   h = SiLU(G) * U                                                 (Sec. 3.3, Sec. 5)
//   y = W4down h                                                    (Sec. 3.3)
// Decode is bound by the bandwidth of loading weights (Sec. 3.3, Sec. 5): each
// lane issues all 128-bit loads of its packed codes before any arithmetic,
// the activation sits in LDS, and rows are reduced with lane butterflies.
//
// Dot products without per-code int->float conversion: a code OR-ed into the
// fraction of binary16 1024.0 reads 1024 + q * 2^j (j = its fraction bit
// position, 4..8).  The activation copy in LDS is pre-scaled by 2^-j per
// position, so v_dot2_f32_f16 over the raw codes yields
//   acc = sum_i q_i x_i + 1024 * sum_i x'_i .
// Per 64-code (2-bit) / 32-code (4-bit) unit u of a row with group scale s and
// zero z:   sum_i s (q_i - z) x_i = s (acc - C_u - z X_u),
// with C_u = 1024 * sum x'_i and X_u = sum x_i staged next to the activation.
//
// Work items: S lanes share one output row; lane s owns the 16-byte units
// u = s, s + S, s + 2S, ... of that row (the S lanes of a row read S
// consecutive units: coalesced), so a wave-item covers 64/S rows.
#pragma once

#include "qmlp_device.h"
#include "qmlp_internal.h"

namespace qmlp {

constexpr int GU_UNIT_BYTES = 8 * 16 + 8;   // LDS bytes per (token, 2-bit unit): x' + (C, X)
constexpr int DN_UNIT_BYTES = 4 * 16 + 8;   // LDS bytes per (token, 4-bit unit): h' + (C, X)

// One-shift forms (the streamed and MFMA kernels): code fields are read where
// they sit in the word, so a word needs one shift.
// 2-bit code pairs of one word, one shift: pair p = (code p, code 8 + p) at
// fraction positions 2 kp, kp = {0, 1, 2, 3, 4, 2, 3, 4}.
__device__ __forceinline__ void extract_w2_s1(uint32_t w, uint32_t e[8], uint32_t mv) {
    const uint32_t r = w >> 6;          // codes 5, 6, 7 -> bits 4-9
    e[0] = magic(w, 0x00030003u, mv);
    e[1] = magic(w, 0x000C000Cu, mv);
    e[2] = magic(w, 0x00300030u, mv);
    e[3] = magic(w, 0x00C000C0u, mv);
    e[4] = magic(w, 0x03000300u, mv);
    e[5] = magic(r, 0x00300030u, mv);
    e[6] = magic(r, 0x00C000C0u, mv);
    e[7] = magic(r, 0x03000300u, mv);
}
__device__ __forceinline__ float w2_s1_scale(int p) {
    const int k = (0x43243210 >> (4 * p)) & 15;
    return __builtin_bit_cast(float, (uint32_t)(127 - 2 * k) << 23);
}

// 4-bit code pairs of one word, one shift: pair p = (code p, code 4 + p) at
// fraction positions {0, 4, 0, 4}.
__device__ __forceinline__ void extract_w4_s1(uint32_t w, uint32_t e[4], uint32_t mv) {
    const uint32_t r = w >> 8;          // codes 2, 3 -> bits 0-7
    e[0] = magic(w, 0x000F000Fu, mv);
    e[1] = magic(w, 0x00F000F0u, mv);
    e[2] = magic(r, 0x000F000Fu, mv);
    e[3] = magic(r, 0x00F000F0u, mv);
}
__device__ __forceinline__ float w4_s1_scale(int p) { return (p & 1) ? 1.0f / 16 : 1.0f; }

// --------------------------------------------------------------- staging
// The activation (x for gate/up, h for down) is staged in LDS pre-scaled per
// fraction position.  Staging is split into a load phase (registers) and a
// convert phase so a kernel can issue these small loads BEFORE its weight
// loads: loads retire in order, so data loaded first is usable while the
// weight stream is still in flight.
//
// x' for 2-bit units [u0, u0+uc): per (token m, unit) eight 16-byte chunks
// (4 code words x 2), chunk c stored at c ^ (unit & 7) so lanes reading
// different units hit different banks; then (C_u, X_u).  One staging "word"
// covers 16 codes of one token (two 16-byte loads).
struct XWord { uint4 lo, hi; };

// Always loads (from word 0 of token 0 when idx has no word or the token is
// padding: a valid address); the convert step zeroes what is not live.
template <int MT>
__device__ __forceinline__ XWord stage_x_load(const uint16_t* x, int M, int d, int u0, int uc,
                                              int idx) {
    const int words = MT * uc * 4;
    const int m = idx / (uc * 4);
    const bool ok = idx < words && m < M;
    const int wl = ok ? idx - m * uc * 4 : 0;
    const uint4* src = reinterpret_cast<const uint4*>(x + (long)(ok ? m : 0) * d + (long)(u0 + (wl >> 2)) * 64 + (wl & 3) * 16);
    return XWord{src[0], src[1]};
}

// Convert one staged word; all lanes of the wave must call it (shuffles).
// SPLIT (group 32 at 2 bits: two groups per 64-code unit) stages (C, X) per
// half unit, two float2 per (token, unit): words 0-1 hold the codes of the
// first group, words 2-3 those of the second.
template <int MT, bool SPLIT = false>
__device__ __forceinline__ void stage_x_store(uint4* xs, float2* cx, int UC, int uc, int M, int idx,
                                              XWord v, uint4* xplain = nullptr) {
    const int words = MT * uc * 4;
    const bool live = idx < words;
    const int m = live ? idx / (uc * 4) : 0;
    const int wl = live ? idx - m * uc * 4 : 0;
    const int ul = wl >> 2, w = wl & 3;
    const bool data = live && m < M;           // padding tokens stage zeros
    const uint32_t xl[4] = {data ? v.lo.x : 0u, data ? v.lo.y : 0u, data ? v.lo.z : 0u, data ? v.lo.w : 0u};
    const uint32_t xh[4] = {data ? v.hi.x : 0u, data ? v.hi.y : 0u, data ? v.hi.z : 0u, data ? v.hi.w : 0u};
    uint32_t pr[8];
    float csum = 0.0f, xsum = 0.0f;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        // pair p = (x[p], x[8 + p]); x[i] is half (i & 1) of word i >> 1
        const uint32_t a16 = (xl[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;
        const uint32_t b16 = (xh[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;
        const float sc = w2_pair_scale(p);
        const uint32_t ha = f2h(h2f(a16) * sc), hb = f2h(h2f(b16) * sc);
        pr[p] = ha | (hb << 16);
        csum += h2f(ha) + h2f(hb);
        xsum += h2f(a16) + h2f(b16);
    }
    csum = group_sum<SPLIT ? 2 : 4>(csum);
    xsum = group_sum<SPLIT ? 2 : 4>(xsum);
    if (live) {
        uint4* dst = xs + (m * UC + ul) * 8;
        dst[(2 * w) ^ (ul & 7)] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        dst[(2 * w + 1) ^ (ul & 7)] = make_uint4(pr[4], pr[5], pr[6], pr[7]);
        if (SPLIT ? (w & 1) == 0 : w == 0)
            cx[SPLIT ? (m * UC + ul) * 2 + (w >> 1) : m * UC + ul] = make_float2(1024.0f * csum, xsum);
        if (xplain) {                          // unscaled copy (single-chunk staging only)
            uint4* dp = xplain + (m * uc + ul) * 8 + w * 2;
            dp[0] = make_uint4(xl[0], xl[1], xl[2], xl[3]);
            dp[1] = make_uint4(xh[0], xh[1], xh[2], xh[3]);
        }
    }
}

// Whole staging of a chunk by the block (load-convert per word).
template <int MT, bool SPLIT = false>
__device__ __forceinline__ void stage_x(uint4* xs, float2* cx, int UC, const uint16_t* x, int M,
                                        int d, int u0, int uc, int tid, int nthreads) {
    const int words = MT * uc * 4;
    for (int idx = tid; idx < ((words + 63) & ~63); idx += nthreads)
        stage_x_store<MT, SPLIT>(xs, cx, UC, uc, M, idx, stage_x_load<MT>(x, M, d, u0, uc, idx));
}

// 3-bit units (stage_x3): x' exactly as stage_x for the 2-bit plane, then a
// second region x'' (MT * UC * 8 chunks after x') for the 1-bit plane: per
// (m, unit) 32 pairs (x[32h+i], x[32h+16+i]) / 256 in binary16, pair p in
// chunk (p/4) ^ (unit & 7).  The (C, X) slot holds C = 1024 (sum x' + 4 sum x''),
// both planes' magic offsets, per unit or per half unit (SPLIT).  Each lane
// writes the 16 halves of its staging word into x'' one by one.
template <int MT, bool SPLIT>
__device__ __forceinline__ void stage_x3_store(uint4* xs, float2* cx, int UC, int uc, int M, int idx,
                                               XWord v) {
    const int words = MT * uc * 4;
    const bool live = idx < words;
    const int m = live ? idx / (uc * 4) : 0;
    const int wl = live ? idx - m * uc * 4 : 0;
    const int ul = wl >> 2, w = wl & 3;
    const bool data = live && m < M;           // padding tokens stage zeros
    const uint32_t xl[4] = {data ? v.lo.x : 0u, data ? v.lo.y : 0u, data ? v.lo.z : 0u, data ? v.lo.w : 0u};
    const uint32_t xh[4] = {data ? v.hi.x : 0u, data ? v.hi.y : 0u, data ? v.hi.z : 0u, data ? v.hi.w : 0u};
    uint32_t pr[8];
    uint16_t x2[16];
    float csum = 0.0f, xsum = 0.0f;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        const uint32_t a16 = (xl[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;     // x[p]
        const uint32_t b16 = (xh[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;     // x[8 + p]
        const float sc = w2_pair_scale(p);
        const uint32_t ha = f2h(h2f(a16) * sc), hb = f2h(h2f(b16) * sc);
        pr[p] = ha | (hb << 16);
        const uint32_t ta = f2h(h2f(a16) * (1.0f / 256)), tb = f2h(h2f(b16) * (1.0f / 256));
        x2[p] = (uint16_t)ta;
        x2[8 + p] = (uint16_t)tb;
        csum += h2f(ha) + h2f(hb) + 4.0f * (h2f(ta) + h2f(tb));
        xsum += h2f(a16) + h2f(b16);
    }
    csum = group_sum<SPLIT ? 2 : 4>(csum);
    xsum = group_sum<SPLIT ? 2 : 4>(xsum);
    if (live) {
        uint4* dst = xs + (m * UC + ul) * 8;
        dst[(2 * w) ^ (ul & 7)] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        dst[(2 * w + 1) ^ (ul & 7)] = make_uint4(pr[4], pr[5], pr[6], pr[7]);
        // word w holds codes 16w..16w+15 of the unit: half h = w/2 of the pairs,
        // the low (w even) or high (w odd) binary16 of each
        uint16_t* d2 = reinterpret_cast<uint16_t*>(xs + MT * UC * 8 + (m * UC + ul) * 8);
        const int h = w >> 1, part = w & 1;
#pragma unroll
        for (int t = 0; t < 16; ++t) {
            const int pi = 16 * h + t;
            d2[(((pi >> 2) ^ (ul & 7)) * 4 + (pi & 3)) * 2 + part] = x2[t];
        }
        if (SPLIT ? (w & 1) == 0 : w == 0)
            cx[SPLIT ? (m * UC + ul) * 2 + (w >> 1) : m * UC + ul] = make_float2(1024.0f * csum, xsum);
    }
}

template <int MT, bool SPLIT>
__device__ __forceinline__ void stage_x3(uint4* xs, float2* cx, int UC, const uint16_t* x, int M,
                                         int d, int u0, int uc, int tid, int nthreads) {
    const int words = MT * uc * 4;
    for (int idx = tid; idx < ((words + 63) & ~63); idx += nthreads)
        stage_x3_store<MT, SPLIT>(xs, cx, UC, uc, M, idx, stage_x_load<MT>(x, M, d, u0, uc, idx));
}

// h' for 4-bit units [u0, u0+uc): per (m, unit) four 16-byte chunks (one per
// code word, 4 pairs), chunk c stored at c ^ ((unit >> 1) & 3); then (C_u, X_u).
// One staging word covers 8 codes of one token (one 16-byte load).
template <int MT>
__device__ __forceinline__ uint4 stage_h_load(const uint16_t* h, int M, int f, int u0, int uc,
                                              int idx) {
    const int words = MT * uc * 4;
    const int m = idx / (uc * 4);
    const bool ok = idx < words && m < M;
    const int wl = ok ? idx - m * uc * 4 : 0;
    return *reinterpret_cast<const uint4*>(h + (long)(ok ? m : 0) * f + (long)(u0 + (wl >> 2)) * 32 + (wl & 3) * 8);
}

template <int MT>
__device__ __forceinline__ void stage_h_store(uint4* hs, float2* cx, int UC, int uc, int M, int idx,
                                              uint4 v) {
    const int words = MT * uc * 4;
    const bool live = idx < words;
    const int m = live ? idx / (uc * 4) : 0;
    const int wl = live ? idx - m * uc * 4 : 0;
    const int ul = wl >> 2, w = wl & 3;
    const bool data = live && m < M;           // padding tokens stage zeros
    const uint32_t hl[4] = {data ? v.x : 0u, data ? v.y : 0u, data ? v.z : 0u, data ? v.w : 0u};
    uint32_t pr[4];
    float csum = 0.0f, xsum = 0.0f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        // pair p = (h[p], h[4 + p])
        const uint32_t a16 = (hl[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;
        const uint32_t b16 = (hl[2 + (p >> 1)] >> (16 * (p & 1))) & 0xFFFFu;
        const float sc = w4_pair_scale(p);
        const uint32_t ha = f2h(h2f(a16) * sc), hb = f2h(h2f(b16) * sc);
        pr[p] = ha | (hb << 16);
        csum += h2f(ha) + h2f(hb);
        xsum += h2f(a16) + h2f(b16);
    }
    csum = group_sum<4>(csum);
    xsum = group_sum<4>(xsum);
    if (live) {
        hs[(m * UC + ul) * 4 + (w ^ ((ul >> 1) & 3))] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        if (w == 0)
            cx[m * UC + ul] = make_float2(1024.0f * csum, xsum);
    }
}

template <int MT>
__device__ __forceinline__ void stage_h(uint4* hs, float2* cx, int UC, const uint16_t* h, int M,
                                        int f, int u0, int uc, int tid, int nthreads) {
    const int words = MT * uc * 4;
    for (int idx = tid; idx < ((words + 63) & ~63); idx += nthreads)
        stage_h_store<MT>(hs, cx, UC, uc, M, idx, stage_h_load<MT>(h, M, f, u0, uc, idx));
}

// --------------------------------------------------------------- gate/up item
// B = code width of gate and up: 2 (W4/W2-GateUp, and uniform W2) or 4
// (uniform W4, the baseline of the precision comparison in Sec. 5.2).  A
// 16-byte unit holds UI = 128/B codes of a row: at 2 bits the activation is
// staged by stage_x (eight chunks per unit), at 4 bits by stage_h (four).
// SPLIT = group 32 at 2 bits (the paper's INT2 grouping, Sec. 3.3 and
// Sec. 4.1): a unit spans two groups, so each carries two metadata words
// and two (C, X) pairs (stage_x<MT, true>).
template <int MT, int S, int MAXJ, int B = 2, bool SPLIT = false, bool TP = (MT == 1 && B == 2)>
struct GuItem {
    static constexpr int NM = SPLIT ? 2 : 1;     // metadata words per unit
    uint4 qg[MAXJ], qu[MAXJ];
    uint2 hg[B == 3 ? MAXJ : 1], hu[B == 3 ? MAXJ : 1];   // 1-bit planes (3 bits)
    uint32_t mg[MAXJ][NM], mu[MAXJ][NM];
    uint32_t bg[4], bu[4];          // LoRA-B row slice, raw binary16
    static constexpr bool TPRE = TP;  // t prefetched with the weights (one token, 2 bits)
    float tg[TPRE ? 4 : 1], tu[TPRE ? 4 : 1];        // the lane's slice of t
    float G[MT], U[MT];
    int row;
    bool ok;
};

// Issue the loads of one gate/up item: S lanes per row, rows row0 + lane/S.
template <int MT, int S, int MAXJ, int B, bool SPLIT, bool TP>
__device__ __forceinline__ void gu_load(GuItem<MT, S, MAXJ, B, SPLIT, TP>& it, const GateUpArgs& a,
                                        int row0, bool active, int lane) {
    static_assert((B == 2 || B == 3 || B == 4) && (!SPLIT || B != 4), "gate/up at 2, 3 or 4 bits");
    constexpr int UI = codes_per_unit(B);
    const int s = lane % S;
    const int U = a.d / UI;
    const int J = (U + S - 1) / S;
    it.row = row0 + lane / S;
    it.ok = active && it.row < a.f;
    const int ng = a.d / a.g;
    const int upg = SPLIT ? 1 : a.g / UI;
    // Loads go out from a clamped, always valid address (unit 0 of row 0 for
    // lanes without work) straight into the slot registers: no select and no
    // conversion touches a loaded value here, since loads retire in order and
    // any use would stall issue until every earlier load of the wave arrived.
    // Values of lanes without work are never used (the compute skips units
    // past the row and the epilogue skips rows past f).
    const long rowc = it.ok ? it.row : 0;
    // 3 bits: a row is its 2-bit plane (d/4 bytes) then its 1-bit plane (d/8).
    const long rstride = B == 3 ? (long)U * 3 / 2 : (long)U;      // in 16-byte units
    const uint4* cg = reinterpret_cast<const uint4*>(a.cg) + rowc * rstride;
    const uint4* cu = reinterpret_cast<const uint4*>(a.cu) + rowc * rstride;
    const uint2* pg = reinterpret_cast<const uint2*>(cg + U);
    const uint2* pu = reinterpret_cast<const uint2*>(cu + U);
    const uint32_t* mg = a.mg + rowc * ng;
    const uint32_t* mu = a.mu + rowc * ng;
#pragma unroll
    for (int i = 0; i < MAXJ; ++i) {
        if (i < J && active) {                     // wave-uniform; unloaded slots are never read
            const int u = s + S * i;
            const int uu = u < U ? u : 0;
            it.qg[i] = load_stream(cg + uu);
            it.qu[i] = load_stream(cu + uu);
            if constexpr (B == 3) {
                it.hg[i] = pg[uu];
                it.hu[i] = pu[uu];
            }
#pragma unroll
            for (int h = 0; h < GuItem<MT, S, MAXJ, B, SPLIT, TP>::NM; ++h) {
                const int gi = SPLIT ? 2 * uu + h : uu / upg;
                it.mg[i][h] = load_stream(mg + gi);
                it.mu[i][h] = load_stream(mu + gi);
            }
        }
    }
    // LoRA-B row slices stay raw binary16 until the epilogue: four loads per
    // lane, branch-free from clamped offsets (with rank 0 the pointers are a
    // readable dummy), so nothing converts them at issue time.
    const int CPL = (a.r + S - 1) / S;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int rc = s * CPL + c;
        const long off = rowc * a.r + ((c < CPL && rc < a.r) ? rc : 0);
        it.bg[c] = a.Bg[off];
        it.bu[c] = a.Bu[off];
    }
    // At one token and 2 bits the lane's slice of t (written by the LoRA-A
    // launch before this one) rides with the weight loads, so the epilogue
    // makes no second trip to memory; with rank 0 a readable dummy (x)
    // stands in.  (With it the 4-bit item measured slower, 8.1 -> 8.6 us per
    // uniform-W4 block, so that item reads t in the epilogue.)
    if constexpr (GuItem<MT, S, MAXJ, B, SPLIT, TP>::TPRE) {
        const float* tp = a.r > 0 ? a.t : reinterpret_cast<const float*>(a.x);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int rc = s * CPL + c;
            const int o = (c < CPL && rc < a.r) ? rc : 0;
            it.tg[c] = tp[o];
            it.tu[c] = tp[a.r + o];
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) it.G[m] = it.U[m] = 0.0f;
}

// Dot products of the item's units that fall in the staged chunk [u0, u0+uc).
template <int MT, int S, int MAXJ, int B, bool SPLIT, bool TP>
__device__ __forceinline__ void gu_accumulate(GuItem<MT, S, MAXJ, B, SPLIT, TP>& it, const uint4* xs,
                                              const float2* cx, int UC, int d, int u0, int uc,
                                              int lane) {
    constexpr int NM = GuItem<MT, S, MAXJ, B, SPLIT, TP>::NM;
    constexpr int UI = codes_per_unit(B);
    const uint32_t mv = 0x64006400u;           // (the standalone kernels keep the literal)
    const int s = lane % S;
    const int J = (d / UI + S - 1) / S;
#pragma unroll
    for (int i = 0; i < MAXJ; ++i) {
        const int u = s + S * i;
        if (i < J && u >= u0 && u < u0 + uc) {
            const int ul = u - u0;
            float ag[NM][MT], au[NM][MT];
            float bg1[B == 3 ? NM : 1][MT], bu1[B == 3 ? NM : 1][MT];   // 1-bit plane sums
#pragma unroll
            for (int h = 0; h < NM; ++h)
#pragma unroll
                for (int m = 0; m < MT; ++m) ag[h][m] = au[h][m] = 0.0f;
#pragma unroll
            for (int h = 0; h < (B == 3 ? NM : 1); ++h)
#pragma unroll
                for (int m = 0; m < MT; ++m) bg1[h][m] = bu1[h][m] = 0.0f;
            uint32_t wg[4] = {it.qg[i].x, it.qg[i].y, it.qg[i].z, it.qg[i].w};
            uint32_t wu[4] = {it.qu[i].x, it.qu[i].y, it.qu[i].z, it.qu[i].w};
            uint32_t mgi[NM], mui[NM];
#pragma unroll
            for (int h = 0; h < NM; ++h) {
                mgi[h] = it.mg[i][h];
                mui[h] = it.mu[i][h];
                pin(mgi[h]);
                pin(mui[h]);
            }
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                pin(wg[w]);
                pin(wu[w]);
            }
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                const int hw = SPLIT ? (w >> 1) : 0;     // the group of code word w
                if constexpr (B == 2 || B == 3) {         // (at 3 bits: the 2-bit plane)
                    uint32_t eg[8], eu[8];
                    extract_w2(wg[w], eg, mv);
                    extract_w2(wu[w], eu, mv);
#pragma unroll
                    for (int m = 0; m < MT; ++m) {
                        const uint4* src = xs + (m * UC + ul) * 8;
                        const uint4 p0 = src[(2 * w) ^ (ul & 7)];
                        const uint4 p1 = src[(2 * w + 1) ^ (ul & 7)];
                        const uint32_t xp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
                        for (int p = 0; p < 8; ++p) {
                            ag[hw][m] = dot2(eg[p], xp[p], ag[hw][m]);
                            au[hw][m] = dot2(eu[p], xp[p], au[hw][m]);
                        }
                    }
                } else {
                    uint32_t eg[4], eu[4];
                    extract_w4(wg[w], eg, mv);
                    extract_w4(wu[w], eu, mv);
#pragma unroll
                    for (int m = 0; m < MT; ++m) {
                        const uint4 p = xs[(m * UC + ul) * 4 + (w ^ ((ul >> 1) & 3))];
                        const uint32_t xp[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
                        for (int c = 0; c < 4; ++c) {
                            ag[0][m] = dot2(eg[c], xp[c], ag[0][m]);
                            au[0][m] = dot2(eu[c], xp[c], au[0][m]);
                        }
                    }
                }
            }
            if constexpr (B == 3) {
                // The 1-bit plane: word h holds the high bits of codes 32h..32h+31
                // (bit i = code 32h+i); pair i = (code 32h+i, code 32h+16+i) meets
                // x'' = x/256 staged in the same pairs (stage_x3).
                const uint4* xs2 = xs + MT * UC * 8;
                uint32_t hgw[2] = {it.hg[i].x, it.hg[i].y};
                uint32_t huw[2] = {it.hu[i].x, it.hu[i].y};
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    pin(hgw[h]);
                    pin(huw[h]);
                }
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int hw = SPLIT ? h : 0;
#pragma unroll
                    for (int cc = 0; cc < 4; ++cc) {
                        uint32_t eg[4], eu[4];
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            eg[q] = bit_pair(hgw[h], 4 * cc + q, mv);
                            eu[q] = bit_pair(huw[h], 4 * cc + q, mv);
                        }
#pragma unroll
                        for (int m = 0; m < MT; ++m) {
                            const uint4 p = xs2[(m * UC + ul) * 8 + ((4 * h + cc) ^ (ul & 7))];
                            const uint32_t xp[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                bg1[hw][m] = dot2(eg[q], xp[q], bg1[hw][m]);
                                bu1[hw][m] = dot2(eu[q], xp[q], bu1[hw][m]);
                            }
                        }
                    }
                }
            }
#pragma unroll
            for (int h = 0; h < NM; ++h) {
                const float sg = h2f(mgi[h] & 0xFFFFu), zg = h2f(mgi[h] >> 16);
                const float su = h2f(mui[h] & 0xFFFFu), zu = h2f(mui[h] >> 16);
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const float2 k = cx[(m * UC + ul) * NM + h];
                    float dg = ag[h][m], du = au[h][m];
                    if constexpr (B == 3) {       // q = q_lo + 4 q_hi; k.x holds both planes' offsets
                        dg += 4.0f * bg1[h][m];
                        du += 4.0f * bu1[h][m];
                    }
                    it.G[m] += sg * (dg - k.x - zg * k.y);
                    it.U[m] += su * (du - k.x - zu * k.y);
                }
            }
        }
    }
}

// LoRA-B on the lane's rank slice, reduction over the S lanes of each row,
// and the epilogue h = SiLU(G) * U (t: [M][2r] fp32, gate ranks then up).
template <int MT, int S, int MAXJ, int B, bool SPLIT, bool TP>
__device__ __forceinline__ void gu_finish(GuItem<MT, S, MAXJ, B, SPLIT, TP>& it, const GateUpArgs& a,
                                          const float* t, uint16_t* h, int lane) {
    const int s = lane % S;
    if (a.r > 0) {
        const int CPL = (a.r + S - 1) / S;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            if (m < a.M) {
                float lg = 0.0f, lu = 0.0f;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int rc = s * CPL + c;
                    if (c < CPL && rc < a.r) {
                        uint32_t bgc = it.bg[c], buc = it.bu[c];
                        pin(bgc);
                        pin(buc);
                        if constexpr (GuItem<MT, S, MAXJ, B, SPLIT, TP>::TPRE) {
                            lg += h2f(bgc) * it.tg[c];
                            lu += h2f(buc) * it.tu[c];
                        } else {
                            lg += h2f(bgc) * t[m * 2 * a.r + rc];
                            lu += h2f(buc) * t[m * 2 * a.r + a.r + rc];
                        }
                    }
                }
                it.G[m] += a.lora_scale * lg;
                it.U[m] += a.lora_scale * lu;
            }
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const float gv = group_sum<S>(it.G[m]);
        const float uv = group_sum<S>(it.U[m]);
        if (it.ok && m < a.M && (m % S) == s) {
            const float hv = gv / (1.0f + __expf(-gv)) * uv;
            h[(long)m * a.f + it.row] = (uint16_t)f2h(hv);
        }
    }
}

// --------------------------------------------------------------- down item
// B = code width of the down projection: 4 (W4/W2-GateUp, uniform W4) or 2
// (uniform W2, Sec. 5.2).  At 4 bits h is staged by stage_h (32 codes per
// unit), at 2 bits by stage_x (64 codes per unit; groups of 64 or 128).
template <int MT, int S, int MAXJ, int B = 4>
struct DnItem {
    uint4 q[MAXJ];
    uint32_t mt[MAXJ];
    float Y[MT];
    int row;
    bool ok;          // this lane's row exists
    bool active;      // the wave holds this item (wave-uniform)
};

template <int MT, int S, int MAXJ, int B>
__device__ __forceinline__ void dn_load(DnItem<MT, S, MAXJ, B>& it, const DownArgs& a, int row0,
                                        bool active, int lane) {
    static_assert(B == 2 || B == 4, "down at 2 or 4 bits");
    constexpr int UI = codes_per_unit(B);
    const int s = lane % S;
    const int U = a.f / UI;
    const int J = (U + S - 1) / S;
    it.row = row0 + lane / S;
    it.ok = active && it.row < a.d;
    it.active = active;
    const int ng = a.f / a.g;
    const int upg = a.g / UI;
    const long rowc = it.ok ? it.row : 0;          // clamped, unselected: see gu_load
    const uint4* cd = reinterpret_cast<const uint4*>(a.cd) + rowc * U;
    const uint32_t* md = a.md + rowc * ng;
#pragma unroll
    for (int i = 0; i < MAXJ; ++i) {
        if (i < J && active) {                     // wave-uniform; unloaded slots are never read
            const int u = s + S * i;
            const int uu = u < U ? u : 0;
            it.q[i] = load_stream(cd + uu);
            it.mt[i] = load_stream(md + uu / upg);
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) it.Y[m] = 0.0f;
}

template <int MT, int S, int MAXJ, int B>
__device__ __forceinline__ void dn_accumulate(DnItem<MT, S, MAXJ, B>& it, const uint4* hs,
                                              const float2* cx, int UC, int f, int u0, int uc,
                                              int lane) {
    constexpr int UI = codes_per_unit(B);
    const uint32_t mv = 0x64006400u;           // (the standalone kernels keep the literal)
    const int s = lane % S;
    const int J = (f / UI + S - 1) / S;
    if (!it.active)
        return;
#pragma unroll
    for (int i = 0; i < MAXJ; ++i) {
        const int u = s + S * i;
        if (i < J && u >= u0 && u < u0 + uc) {
            const int ul = u - u0;
            float acc[MT];
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[m] = 0.0f;
            uint32_t wv[4] = {it.q[i].x, it.q[i].y, it.q[i].z, it.q[i].w};
            uint32_t mti = it.mt[i];
#pragma unroll
            for (int w = 0; w < 4; ++w)
                pin(wv[w]);
            pin(mti);
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                if constexpr (B == 4) {
                    uint32_t e[4];
                    extract_w4(wv[w], e, mv);
#pragma unroll
                    for (int m = 0; m < MT; ++m) {
                        const uint4 p = hs[(m * UC + ul) * 4 + (w ^ ((ul >> 1) & 3))];
                        acc[m] = dot2(e[0], p.x, acc[m]);
                        acc[m] = dot2(e[1], p.y, acc[m]);
                        acc[m] = dot2(e[2], p.z, acc[m]);
                        acc[m] = dot2(e[3], p.w, acc[m]);
                    }
                } else {
                    uint32_t e[8];
                    extract_w2(wv[w], e, mv);
#pragma unroll
                    for (int m = 0; m < MT; ++m) {
                        const uint4* src = hs + (m * UC + ul) * 8;
                        const uint4 p0 = src[(2 * w) ^ (ul & 7)];
                        const uint4 p1 = src[(2 * w + 1) ^ (ul & 7)];
                        const uint32_t hp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
                        for (int p = 0; p < 8; ++p) acc[m] = dot2(e[p], hp[p], acc[m]);
                    }
                }
            }
            const float sc = h2f(mti & 0xFFFFu), zc = h2f(mti >> 16);
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const float2 k = cx[m * UC + ul];
                it.Y[m] += sc * (acc[m] - k.x - zc * k.y);
            }
        }
    }
}

template <int MT, int S, int MAXJ, int B>
__device__ __forceinline__ void dn_finish(DnItem<MT, S, MAXJ, B>& it, const DownArgs& a, int lane) {
    const int s = lane % S;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const float v = group_sum<S>(it.Y[m]);
        if (it.ok && m < a.M && (m % S) == s)
            a.y[(long)m * a.d + it.row] = (uint16_t)f2h(v);
    }
}


// --------------------------------------------------------------- fused-kernel items
// Straight-line load sequences for the fused layer kernel: exactly the same
// number of loads on every lane and path, so the wait before each use covers
// exactly the loads issued before it.  Lanes without work read a clamped,
// valid address and their values are never used.
//
// Scale/zero metadata is loaded WIDE: the rows of a wave-item have
// consecutive metadata words, which the wave pulls in with 16-byte loads
// (one or two instructions instead of one 4-byte load per slot) and parks in
// a per-wave LDS area; each lane then reads its groups' words from LDS.
template <int MT, int S, int MAXJ, int KMETA>
struct FGuItem {
    uint4 qg[MAXJ], qu[MAXJ];
    uint4 meta[KMETA];           // metadata chunks, gate rows then up rows (KMETA per lane)
    uint32_t bg[2], bu[2];       // LoRA-B row slice, raw binary16 (up to 4 halves)
    float G[MT], U[MT];
    int row, row0;
    bool ok;
};

// Loads: metadata chunks first (they retire first), then codes, then LoRA-B.
template <int MT, int S, int MAXJ, int KMETA, int WIN = 0>
__device__ __forceinline__ void fgu_load(FGuItem<MT, S, MAXJ, KMETA>& it, const GateUpArgs& a, int row0,
                                         int lane) {
    constexpr int RPW = 64 / S;
    const int s = lane % S;
    const int U = a.d / 64;
    const int ng = a.d / a.g;
    it.row0 = row0;
    it.row = row0 + lane / S;
    it.ok = it.row < a.f;
    const long rowc = it.ok ? it.row : 0;
    // metadata of rows row0 .. row0+RPW-1: RPW*ng words per matrix, 16-byte
    // aligned (row0 is a multiple of RPW and RPW*ng*4 a multiple of 16)
    const int chunks = RPW * ng / 4;                       // per matrix
    const uint4* mg = reinterpret_cast<const uint4*>(a.mg + (long)row0 * ng);
    const uint4* mu = reinterpret_cast<const uint4*>(a.mu + (long)row0 * ng);
#pragma unroll
    for (int k = 0; k < KMETA; ++k) {
        const int c = lane + 64 * k;                       // chunk over [gate | up]
        const uint4* src = c < chunks ? mg + c : (c < 2 * chunks ? mu + (c - chunks) : mg);
        it.meta[k] = load_stream(src);
    }
    const uint4* cg = reinterpret_cast<const uint4*>(a.cg) + rowc * U;
    const uint4* cu = reinterpret_cast<const uint4*>(a.cu) + rowc * U;
#pragma unroll
    for (int i = 0; i < MAXJ; ++i) {
        const int u = s + S * i;
        const int uu = u < U ? u : 0;
        if constexpr (WIN > 0) {
            if (2 * i + KMETA >= WIN)
                vm_window<WIN - 2>();
        }
        it.qg[i] = load_stream(cg + uu);
        it.qu[i] = load_stream(cu + uu);
    }
    // LoRA-B: lane s takes ranks [s*CPL, s*CPL + CPL), one load per matrix
    const int CPL = (a.r + S - 1) / S;
    const long off = rowc * a.r + (s * CPL < a.r ? s * CPL : 0);
    if (CPL <= 1) {
        it.bg[0] = a.Bg[off];
        it.bu[0] = a.Bu[off];
    } else if (CPL == 2) {
        it.bg[0] = *reinterpret_cast<const uint32_t*>(a.Bg + off);
        it.bu[0] = *reinterpret_cast<const uint32_t*>(a.Bu + off);
    } else {
        const uint2 vg = *reinterpret_cast<const uint2*>(a.Bg + off);
        const uint2 vu = *reinterpret_cast<const uint2*>(a.Bu + off);
        it.bg[0] = vg.x; it.bg[1] = vg.y;
        it.bu[0] = vu.x; it.bu[1] = vu.y;
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) it.G[m] = it.U[m] = 0.0f;
}

// Park the metadata chunks in the wave's LDS area (gate rows, then up rows).
template <int MT, int S, int MAXJ, int KMETA>
__device__ __forceinline__ void fgu_meta_to_lds(const FGuItem<MT, S, MAXJ, KMETA>& it, const GateUpArgs& a,
                                                uint4* wmeta, int lane) {
    constexpr int RPW = 64 / S;
    const int chunks = RPW * (a.d / a.g) / 4;
#pragma unroll
    for (int k = 0; k < KMETA; ++k) {
        const int c = lane + 64 * k;
        if (c < 2 * chunks)
            wmeta[c] = it.meta[k];
    }
}

// Branch-free over the unit slots (a slot past the row's last unit re-reads
// unit 0 and adds it with scale 0).  At one token the eight 16-byte x' reads
// of slot i + 1 are issued before slot i is computed (the compiler would
// otherwise wait on each read in turn).
template <int MT, int S, int MAXJ, int KMETA>
__device__ __forceinline__ void fgu_slot(FGuItem<MT, S, MAXJ, KMETA>& it, int i, int ul, bool valid,
                                         const uint4 (&xv)[MT][8], const float2* cx, int UC, int ng,
                                         int gsh, const uint32_t* wmeta, int r) {
    const uint32_t mv = MT >= 4 ? 0x64006400u : magic_vgpr();   // a VGPR, except at 4 tokens
    constexpr int RPW = 64 / S;
    float ag[MT], au[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) ag[m] = au[m] = 0.0f;
    uint32_t wg[4] = {it.qg[i].x, it.qg[i].y, it.qg[i].z, it.qg[i].w};
    uint32_t wu[4] = {it.qu[i].x, it.qu[i].y, it.qu[i].z, it.qu[i].w};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        pin(wg[w]);
        pin(wu[w]);
    }
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        uint32_t eg[8], eu[8];
        extract_w2(wg[w], eg, mv);
        extract_w2(wu[w], eu, mv);
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            const uint4 p0 = xv[m][2 * w], p1 = xv[m][2 * w + 1];
            const uint32_t xp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                ag[m] = dot2(eg[p], xp[p], ag[m]);
                au[m] = dot2(eu[p], xp[p], au[m]);
            }
        }
    }
    const uint32_t mgi = wmeta[r * ng + (ul >> gsh)];
    const uint32_t mui = wmeta[(RPW + r) * ng + (ul >> gsh)];
    const float sg = valid ? h2f(mgi & 0xFFFFu) : 0.0f, zg = h2f(mgi >> 16);
    const float su = valid ? h2f(mui & 0xFFFFu) : 0.0f, zu = h2f(mui >> 16);
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const float2 k = cx[m * UC + ul];
        it.G[m] += sg * (ag[m] - k.x - zg * k.y);
        it.U[m] += su * (au[m] - k.x - zu * k.y);
    }
}

template <int MT>
__device__ __forceinline__ void fgu_read_x(uint4 (&xv)[MT][8], const uint4* xs, int UC, int ul) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const uint4* src = xs + (m * UC + ul) * 8;
#pragma unroll
        for (int c = 0; c < 8; ++c) xv[m][c] = src[c ^ (ul & 7)];
    }
}

template <int MT, int S, int MAXJ, int KMETA>
__device__ __forceinline__ void fgu_accumulate(FGuItem<MT, S, MAXJ, KMETA>& it, const uint4* xs,
                                               const float2* cx, int UC, int d, int g,
                                               const uint32_t* wmeta, int lane) {
    const uint32_t mv = MT >= 4 ? 0x64006400u : magic_vgpr();   // a VGPR, except at 4 tokens
    const int s = lane % S, r = lane / S;
    const int U = d / 64, ng = d / g, gsh = g == 128 ? 1 : 0;   // units of 64 per group: 1 << gsh
    if constexpr (MT == 1) {
        // two buffers in turn: the reads of slot i + 1 go out before slot i
        uint4 bx[2][1][8];
        fgu_read_x<1>(bx[0], xs, UC, s < U ? s : 0);
#pragma unroll
        for (int i = 0; i < MAXJ; ++i) {
            const int u = s + S * i, un = u + S;
            const bool valid = u < U;
            if (i + 1 < MAXJ)
                fgu_read_x<1>(bx[(i + 1) & 1], xs, UC, un < U ? un : 0);
#pragma unroll
            for (int c = 0; c < 8; ++c) pin4(bx[i & 1][0][c]);
            fgu_slot(it, i, valid ? u : 0, valid, bx[i & 1], cx, UC, ng, gsh, wmeta, r);
        }
    } else if constexpr (MT == 2) {
#pragma unroll
        for (int i = 0; i < MAXJ; ++i) {
            const int u = s + S * i;
            const bool valid = u < U;
            uint4 xv[MT][8];
            fgu_read_x<MT>(xv, xs, UC, valid ? u : 0);
            fgu_slot(it, i, valid ? u : 0, valid, xv, cx, UC, ng, gsh, wmeta, r);
        }
    } else {
        // four tokens: read x' word by word (a slot's 32 reads would not fit
        // in registers next to the weights)
        constexpr int RPW = 64 / S;
#pragma unroll
        for (int i = 0; i < MAXJ; ++i) {
            const int u = s + S * i;
            const bool valid = u < U;
            const int ul = valid ? u : 0;
            float ag[MT], au[MT];
#pragma unroll
            for (int m = 0; m < MT; ++m) ag[m] = au[m] = 0.0f;
            uint32_t wg[4] = {it.qg[i].x, it.qg[i].y, it.qg[i].z, it.qg[i].w};
            uint32_t wu[4] = {it.qu[i].x, it.qu[i].y, it.qu[i].z, it.qu[i].w};
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                pin(wg[w]);
                pin(wu[w]);
            }
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                uint32_t eg[8], eu[8];
                extract_w2(wg[w], eg, mv);
                extract_w2(wu[w], eu, mv);
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const uint4* src = xs + (m * UC + ul) * 8;
                    const uint4 p0 = src[(2 * w) ^ (ul & 7)];
                    const uint4 p1 = src[(2 * w + 1) ^ (ul & 7)];
                    const uint32_t xp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
                    for (int p = 0; p < 8; ++p) {
                        ag[m] = dot2(eg[p], xp[p], ag[m]);
                        au[m] = dot2(eu[p], xp[p], au[m]);
                    }
                }
            }
            const uint32_t mgi = wmeta[r * ng + (ul >> gsh)];
            const uint32_t mui = wmeta[(RPW + r) * ng + (ul >> gsh)];
            const float sg = valid ? h2f(mgi & 0xFFFFu) : 0.0f, zg = h2f(mgi >> 16);
            const float su = valid ? h2f(mui & 0xFFFFu) : 0.0f, zu = h2f(mui >> 16);
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const float2 k = cx[m * UC + ul];
                it.G[m] += sg * (ag[m] - k.x - zg * k.y);
                it.U[m] += su * (au[m] - k.x - zu * k.y);
            }
        }
    }
}

// LoRA-B, row reduction, h = SiLU(G) * U.  h is published to the other
// compute units as tagged 32-bit words (binary16 value | tag << 16) with
// device-coherent stores: a consumer that reads the current tag has read the
// current value (an aligned 32-bit store is seen whole), so no flag or
// completion wait is needed.
template <int MT, int S, int MAXJ, int KMETA>
__device__ __forceinline__ void fgu_finish(FGuItem<MT, S, MAXJ, KMETA>& it, const GateUpArgs& a,
                                           const float* t, uint32_t* h32, uint32_t tag, int lane) {
    const int s = lane % S;
    if (a.r > 0) {
        const int CPL = (a.r + S - 1) / S;
        uint32_t b0 = it.bg[0], b1 = it.bg[1], c0 = it.bu[0], c1 = it.bu[1];
        pin(b0); pin(b1); pin(c0); pin(c1);
        const uint32_t bgw[2] = {b0, b1}, buw[2] = {c0, c1};
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            if (m < a.M) {
                float lg = 0.0f, lu = 0.0f;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const int rc = s * CPL + c;
                    if (c < CPL && rc < a.r) {
                        lg += h2f(bgw[c >> 1] >> (16 * (c & 1))) * t[m * 2 * a.r + rc];
                        lu += h2f(buw[c >> 1] >> (16 * (c & 1))) * t[m * 2 * a.r + a.r + rc];
                    }
                }
                it.G[m] += a.lora_scale * lg;
                it.U[m] += a.lora_scale * lu;
            }
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const float gv = group_sum<S>(it.G[m]);
        const float uv = group_sum<S>(it.U[m]);
        if (it.ok && m < a.M && (m % S) == s) {
            const float hv = gv / (1.0f + __expf(-gv)) * uv;
            __hip_atomic_store(h32 + (long)m * a.f + it.row, f2h(hv) | (tag << 16),
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

template <int MT, int S, int MAXJ>
struct FDnItem {
    uint4 q[MAXJ];
    uint32_t e[MAXJ][4][4];      // codes unpacked to binary16 pairs (off the critical path)
    uint4 meta;                  // one 16-byte metadata chunk per lane
    float Y[MT];
    int row, row0;
    bool ok, active;
};

// Unpack the item's codes into binary16 pairs while waiting for h.
template <int MT, int S, int MAXJ>
__device__ __forceinline__ void fdn_extract(FDnItem<MT, S, MAXJ>& it) {
    const uint32_t mv = MT >= 4 ? 0x64006400u : magic_vgpr();   // a VGPR, except at 4 tokens
#pragma unroll
    for (int i = 0; i < MAXJ; ++i) {
        uint32_t wv[4] = {it.q[i].x, it.q[i].y, it.q[i].z, it.q[i].w};
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            extract_w4(wv[w], it.e[i][w], mv);
#pragma unroll
            for (int p = 0; p < 4; ++p) pin(it.e[i][w][p]);    // computed here, not at use
        }
    }
}

template <int MT, int S, int MAXJ, int WIN = 0>
__device__ __forceinline__ void fdn_load(FDnItem<MT, S, MAXJ>& it, const DownArgs& a, int row0,
                                         bool active, int lane) {
    constexpr int RPW = 64 / S;
    const int s = lane % S;
    const int U = a.f / 32;
    const int ng = a.f / a.g;
    it.row0 = row0;
    it.row = row0 + lane / S;
    it.ok = active && it.row < a.d;
    it.active = active;
    const long rowc = it.ok ? it.row : 0;
    const int chunks = RPW * ng / 4;                       // <= 64 (checked by the planner)
    const uint4* md = reinterpret_cast<const uint4*>(a.md + (long)(active ? row0 : 0) * ng);
    it.meta = load_stream(md + (lane < chunks ? lane : 0));
    const uint4* cd = reinterpret_cast<const uint4*>(a.cd) + rowc * U;
#pragma unroll
    for (int i = 0; i < MAXJ; ++i) {
        const int u = s + S * i;
        if constexpr (WIN > 0)
            vm_window<WIN - 1>();               // the wave's earlier loads count too
        it.q[i] = load_stream(cd + (u < U ? u : 0));
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) it.Y[m] = 0.0f;
}

template <int MT, int S, int MAXJ>
__device__ __forceinline__ void fdn_meta_to_lds(const FDnItem<MT, S, MAXJ>& it, const DownArgs& a,
                                                uint4* wmeta, int lane) {
    constexpr int RPW = 64 / S;
    if (lane < RPW * (a.f / a.g) / 4)
        wmeta[lane] = it.meta;
}

// Branch-free over the unit slots like fgu_accumulate (an inactive item is
// skipped by a wave-uniform branch); at one token the h' reads of slot i + 1
// are in flight while slot i is computed.
template <int MT, int S, int MAXJ>
__device__ __forceinline__ void fdn_read_h(uint4 (&hv)[MT][4], const uint4* hs, int UC, int ul) {
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int w = 0; w < 4; ++w) hv[m][w] = hs[(m * UC + ul) * 4 + (w ^ ((ul >> 1) & 3))];
}

template <int MT, int S, int MAXJ>
__device__ __forceinline__ void fdn_slot(FDnItem<MT, S, MAXJ>& it, int i, int ul, bool valid,
                                         const uint4 (&hv)[MT][4], const float2* cx, int UC, int ng,
                                         int gsh, const uint32_t* wmeta, int r) {
    float acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
#pragma unroll
        for (int m = 0; m < MT; ++m) {
            const uint4 p = hv[m][w];
            acc[m] = dot2(it.e[i][w][0], p.x, acc[m]);
            acc[m] = dot2(it.e[i][w][1], p.y, acc[m]);
            acc[m] = dot2(it.e[i][w][2], p.z, acc[m]);
            acc[m] = dot2(it.e[i][w][3], p.w, acc[m]);
        }
    }
    const uint32_t mti = wmeta[r * ng + (ul >> gsh)];
    const float sc = valid ? h2f(mti & 0xFFFFu) : 0.0f, zc = h2f(mti >> 16);
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const float2 k = cx[m * UC + ul];
        it.Y[m] += sc * (acc[m] - k.x - zc * k.y);
    }
}

template <int MT, int S, int MAXJ>
__device__ __forceinline__ void fdn_accumulate(FDnItem<MT, S, MAXJ>& it, const uint4* hs,
                                               const float2* cx, int UC, int f, int g,
                                               const uint32_t* wmeta, int lane) {
    const int s = lane % S, r = lane / S;
    const int U = f / 32, ng = f / g, gsh = g == 128 ? 2 : 1;   // units of 32 per group: 1 << gsh
    if (!it.active)
        return;
    if constexpr (MT == 1) {
        uint4 bh[2][1][4];
        fdn_read_h<1, S, MAXJ>(bh[0], hs, UC, s < U ? s : 0);
#pragma unroll
        for (int i = 0; i < MAXJ; ++i) {
            const int u = s + S * i, un = u + S;
            const bool valid = u < U;
            if (i + 1 < MAXJ)
                fdn_read_h<1, S, MAXJ>(bh[(i + 1) & 1], hs, UC, un < U ? un : 0);
#pragma unroll
            for (int w = 0; w < 4; ++w) pin4(bh[i & 1][0][w]);
            fdn_slot(it, i, valid ? u : 0, valid, bh[i & 1], cx, UC, ng, gsh, wmeta, r);
        }
    } else {
#pragma unroll
        for (int i = 0; i < MAXJ; ++i) {
            const int u = s + S * i;
            const bool valid = u < U;
            const int ul = valid ? u : 0;
            float acc[MT];
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[m] = 0.0f;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const uint4 p = hs[(m * UC + ul) * 4 + (w ^ ((ul >> 1) & 3))];
                    acc[m] = dot2(it.e[i][w][0], p.x, acc[m]);
                    acc[m] = dot2(it.e[i][w][1], p.y, acc[m]);
                    acc[m] = dot2(it.e[i][w][2], p.z, acc[m]);
                    acc[m] = dot2(it.e[i][w][3], p.w, acc[m]);
                }
            }
            const uint32_t mti = wmeta[r * ng + (ul >> gsh)];
            const float sc = valid ? h2f(mti & 0xFFFFu) : 0.0f, zc = h2f(mti >> 16);
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const float2 k = cx[m * UC + ul];
                it.Y[m] += sc * (acc[m] - k.x - zc * k.y);
            }
        }
    }
}

template <int MT, int S, int MAXJ>
__device__ __forceinline__ void fdn_finish(FDnItem<MT, S, MAXJ>& it, const DownArgs& a, int lane) {
    const int s = lane % S;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const float v = group_sum<S>(it.Y[m]);
        if (it.ok && m < a.M && (m % S) == s)
            a.y[(long)m * a.d + it.row] = (uint16_t)f2h(v);
    }
}

// Device-coherent read of one staging word of h (8 values) from the tagged
// words written by fgu_finish: two 128-bit buffer loads with the
// device-scope cache policy (sc1).  *ok is false while any of the 8 words
// still carries another call's tag.
template <int MT>
__device__ __forceinline__ uint4 stage_h_load_tagged(__amdgpu_buffer_rsrc_t hrs, int f, int M,
                                                     int uc, int idx, uint32_t tag, bool& ok) {
    const int words = MT * uc * 4;
    const int m = idx / (uc * 4);
    const bool live = idx < words && m < M;
    const int wl = live ? idx - m * uc * 4 : 0;
    const int off = (int)(((long)(live ? m : 0) * f + (long)(wl >> 2) * 32 + (wl & 3) * 8) * 4);
    const u32x4 a = __builtin_amdgcn_raw_buffer_load_b128(hrs, off, 0, 16 /* sc1 */);
    const u32x4 b = __builtin_amdgcn_raw_buffer_load_b128(hrs, off + 16, 0, 16 /* sc1 */);
    const uint32_t tt = tag * 0x10001u;
    ok = ((a.x >> 16) | (a.y & 0xFFFF0000u)) == tt && ((a.z >> 16) | (a.w & 0xFFFF0000u)) == tt &&
         ((b.x >> 16) | (b.y & 0xFFFF0000u)) == tt && ((b.z >> 16) | (b.w & 0xFFFF0000u)) == tt;
    return make_uint4((a.x & 0xFFFFu) | (a.y << 16), (a.z & 0xFFFFu) | (a.w << 16),
                      (b.x & 0xFFFFu) | (b.y << 16), (b.z & 0xFFFFu) | (b.w << 16));
}

// LoRA-A for the fused kernel, split so its loads go out early and the
// arithmetic runs later: one row c of [A_g; A_u] in KA 8-element chunks per
// lane (d <= 512 * KA); x is read from the plain copy staged in LDS.
template <int KA>
struct LoraRow {
    uint4 av[KA];
};

template <int KA>
__device__ __forceinline__ void lora_a_load(LoraRow<KA>& lr, const uint16_t* Ag, const uint16_t* Au,
                                            int d, int r, int c, int lane) {
    const uint16_t* a = c < r ? Ag + (long)c * d : Au + (long)(c - r) * d;
    const int nch = d / 8;
#pragma unroll
    for (int k = 0; k < KA; ++k) {
        const int ch = lane + 64 * k;
        lr.av[k] = *reinterpret_cast<const uint4*>(a + (ch < nch ? ch : 0) * 8);
    }
}

// t[m][c], published as tagged 64-bit words (fp32 bits | tag << 32) with
// device-coherent stores into one private copy per block (t64 + b * 256,
// [4][2r] words each): every block then polls lines no other block reads,
// instead of all blocks polling the same few lines.
// xplain: the staged activation, [MT][d] binary16 in LDS.
template <int MT, int KA>
__device__ __forceinline__ void lora_a_finish(const LoraRow<KA>& lr, const uint4* xplain, int M,
                                              int d, int r, int c, unsigned long long* t64,
                                              uint32_t tag, int blocks, int lane) {
    const int nch = d / 8;
    float acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = 0.0f;
#pragma unroll
    for (int k = 0; k < KA; ++k) {
        const int ch = lane + 64 * k;
        if (ch < nch) {
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const uint4 xv = xplain[m * nch + ch];
                acc[m] = dot2(lr.av[k].x, xv.x, acc[m]);
                acc[m] = dot2(lr.av[k].y, xv.y, acc[m]);
                acc[m] = dot2(lr.av[k].z, xv.z, acc[m]);
                acc[m] = dot2(lr.av[k].w, xv.w, acc[m]);
            }
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const float v = group_sum<64>(acc[m]);
        const unsigned long long word =
            (unsigned long long)__float_as_uint(v) | ((unsigned long long)tag << 32);
        if (m < M)
            for (int blk = lane; blk < blocks; blk += 64)
                __hip_atomic_store(t64 + (long)blk * 256 + m * 2 * r + c, word, __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
    }
}

// --------------------------------------------------------------- LoRA-A row
// t[m][c] = sum_i A[c][i] x[m][i] for one row c of [A_g; A_u], by one wave.
// Every load of the row is issued before the first multiply (KA = most
// 8-element chunks per lane, d <= 512 * KA): in a memory system saturated by
// weight streams a load-use chain would pay one queueing delay per step.
template <int MT, int KA>
__device__ __forceinline__ void lora_a_row(const uint16_t* Ag, const uint16_t* Au,
                                           const uint16_t* x, int M, int d, int r, int c,
                                           float* t, int lane) {
    const uint16_t* a = c < r ? Ag + (long)c * d : Au + (long)(c - r) * d;
    const int nch = d / 8;
    float acc[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) acc[m] = 0.0f;
    for (int base = 0; base < nch; base += 64 * KA) {
        uint4 av[KA], xv[KA][MT];
#pragma unroll
        for (int k = 0; k < KA; ++k) {
            const int ch = base + lane + 64 * k;
            const int cc = ch < nch ? ch : 0;
            av[k] = *reinterpret_cast<const uint4*>(a + cc * 8);
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                const int mm = m < M ? m : 0;
                xv[k][m] = *reinterpret_cast<const uint4*>(x + (long)mm * d + cc * 8);
            }
        }
#pragma unroll
        for (int k = 0; k < KA; ++k) {
            if (base + lane + 64 * k < nch) {
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    acc[m] = dot2(av[k].x, xv[k][m].x, acc[m]);
                    acc[m] = dot2(av[k].y, xv[k][m].y, acc[m]);
                    acc[m] = dot2(av[k].z, xv[k][m].z, acc[m]);
                    acc[m] = dot2(av[k].w, xv[k][m].w, acc[m]);
                }
            }
        }
    }
#pragma unroll
    for (int m = 0; m < MT; ++m) {
        const float v = group_sum<64>(acc[m]);
        if (lane == 0 && m < M)   // device-coherent: read by other compute units
            __hip_atomic_store(t + m * 2 * r + c, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// The call counter of a control block advances by one.  Called by one lane
// of one workgroup of a launch that runs, in stream order, after every
// reader of the counter in the call and before the next call's first one.
__device__ __forceinline__ void advance_call_counter(unsigned* c) {
    const unsigned e = __hip_atomic_load(c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(c, e + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One row of [A_g; A_u] against one token: the dot over d (every load of
// the row issued before the first multiply, as in lora_a_row), summed over
// the wave; every lane returns the sum.
template <int KA>
__device__ __forceinline__ float lora_a_dot(const uint16_t* a, const uint16_t* x, int d, int lane) {
    const int nch = d / 8;
    float acc = 0.0f;
    for (int base = 0; base < nch; base += 64 * KA) {
        uint4 av[KA], xv[KA];
#pragma unroll
        for (int k = 0; k < KA; ++k) {
            const int ch = base + lane + 64 * k;
            const int cc = ch < nch ? ch : 0;
            av[k] = *reinterpret_cast<const uint4*>(a + cc * 8);
            xv[k] = *reinterpret_cast<const uint4*>(x + cc * 8);
        }
#pragma unroll
        for (int k = 0; k < KA; ++k) {
            if (base + lane + 64 * k < nch) {
                acc = dot2(av[k].x, xv[k].x, acc);
                acc = dot2(av[k].y, xv[k].y, acc);
                acc = dot2(av[k].z, xv[k].z, acc);
                acc = dot2(av[k].w, xv[k].w, acc);
            }
        }
    }
    return group_sum<64>(acc);
}

}  // namespace qmlp

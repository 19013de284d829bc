// Building blocks of the persistent decode kernels (M = 1, binary16) on
// gfx950: the work split over 8 XCDs of 32 workgroups, tagged hand-off
// words, and the gate/up and down wave-items that hold a layer's weights in
// registers (the MLP block of Sec. 3.1 Eq. (1), Sec. 3.3, Sec. 4.2).
//
// Hand-offs carry their own validity: each published value sits in one
// aligned word with a 16-bit tag that changes with every layer step (32-bit
// words: binary16 | tag << 16; 64-bit words: fp32 bits | tag << 32).
// XCD-local words are written with plain stores and polled with sc0|nt
// loads (they miss the CU's L1 and hit the XCD's L2); cross-XCD words are
// written and polled device-coherent (sc1).  Every wait is bounded.
#pragma once
#include "decode_common.h"
#include "decode_launch.h"

namespace qmlp {

namespace {

constexpr int SX = 8;                     // XCDs
constexpr int SB = 32;                    // workgroups per XCD
constexpr int SGRID = SX * SB;
constexpr int SCW = 6;                    // weight / compute waves
constexpr int SPW = 2;                    // polling waves
constexpr int SPT = SPW * 64;             // polling threads
constexpr int STHREADS = (SCW + SPW) * 64;
constexpr unsigned kStackSpin = 1u << 17;
constexpr int KXW = 2;                    // activation staging words per polling thread (max)
constexpr int KHW = 2;                    // h staging words per polling thread (max)

// Control words (uint32 index into the stack's control block).
constexpr int C_SEQ = 0, C_DONE = 32, C_ERR = 64, C_XC = 96;

// Cache policy bits of the hand-off loads (bit 31: volatile to the compiler).
constexpr int POL_INTRA = (int)0x80000003u;   // sc0 | nt: through to this XCD's L2
constexpr int POL_CROSS = (int)0x80000010u;   // sc1: device-coherent

__device__ __forceinline__ uint32_t stag(uint32_t s) { return s % 65535u + 1u; }
// 32-bit tag of a step, for the 64-bit hand-off words (never 0)
__device__ __forceinline__ uint32_t ltag32(uint32_t step) { return step % 0xFFFFFFFFu + 1u; }

// Compiler-only fence: the next layer's weight loads are not hoisted above
// the arithmetic on the current layer's registers (which would keep both
// register sets live).
__device__ __forceinline__ void sk_order() { __asm__ volatile("" ::: "memory"); }

__device__ __forceinline__ void st_intra32(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void st_intra64(unsigned long long* p, unsigned long long v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void st_cross64(unsigned long long* p, unsigned long long v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

struct StackLayer {
    const uint32_t *cg, *mg, *cu, *mu, *cd, *md;   // packed codes and (scale | zero << 16) words
    const uint16_t *Bg, *Bu, *Ag, *Au;             // LoRA factors, binary16
    float lora_scale;
};

// Poll K 16-byte words at byte offsets off[k] (only those whose bit is set
// in `valid`) until each shows `tag`: in the high half of every 32-bit word
// (k < K64), or in the high word of both 64-bit halves (k >= K64).  Loads of
// one round go out together; only words still pending are read again.
// sk_poll_issue sends the first round and sk_poll_finish checks it and polls
// on, so several polls can have their first round in flight at once.
template <int K, int POL>
__device__ __forceinline__ void sk_poll_issue(__amdgpu_buffer_rsrc_t rs, const int (&off)[K], uint32_t valid,
                                              u32x4 (&v)[K]) {
#pragma unroll
    for (int k = 0; k < K; ++k)
        if (valid & (1u << k)) v[k] = __builtin_amdgcn_raw_buffer_load_b128(rs, off[k], 0, POL);
}

template <int K, int K64>
__device__ __forceinline__ uint32_t sk_poll_check(const u32x4 (&v)[K], uint32_t pending, uint32_t tag) {
#pragma unroll
    for (int k = 0; k < K; ++k) {
        if (pending & (1u << k)) {
            const bool ok = k >= K64 ? (v[k].y == tag && v[k].w == tag)
                                     : ((v[k].x >> 16) == tag && (v[k].y >> 16) == tag &&
                                        (v[k].z >> 16) == tag && (v[k].w >> 16) == tag);
            if (ok) pending &= ~(1u << k);
        }
    }
    return pending;
}

template <int K, int K64, int POL>
__device__ __forceinline__ bool sk_poll_finish(__amdgpu_buffer_rsrc_t rs, const int (&off)[K], uint32_t valid,
                                               u32x4 (&v)[K], uint32_t tag) {
    uint32_t pending = sk_poll_check<K, K64>(v, valid, tag);
    for (unsigned it = 0; pending != 0u && it < kStackSpin; ++it) {
        __builtin_amdgcn_s_sleep(1);
        sk_poll_issue<K, POL>(rs, off, pending, v);
        pending = sk_poll_check<K, K64>(v, pending, tag);
    }
    return pending == 0u;
}

template <int K, int K64, int POL>
__device__ __forceinline__ bool sk_poll(__amdgpu_buffer_rsrc_t rs, const int (&off)[K], uint32_t valid,
                                        u32x4 (&v)[K], uint32_t tag, bool skip) {
    if (skip)
        return false;
    sk_poll_issue<K, POL>(rs, off, valid, v);
    return sk_poll_finish<K, K64, POL>(rs, off, valid, v, tag);
}

// One staging word of h: 8 binary16 values h[8w .. 8w+8) of this XCD's
// slice into the h' layout of the down units, chunk-major hs[c * HS + ul]
// for chunk c (0..3) of 32-code unit ul = w / 4; and per unit
// (1024 sum h', sum h).
template <int HS>
__device__ __forceinline__ void sk_stage_h(uint4* hs, float2* cx, const u32x4* v, bool valid, int w) {
    uint32_t hv[8];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        hv[4 * q + 0] = valid ? v[q].x & 0xFFFFu : 0u;
        hv[4 * q + 1] = valid ? v[q].y & 0xFFFFu : 0u;
        hv[4 * q + 2] = valid ? v[q].z & 0xFFFFu : 0u;
        hv[4 * q + 3] = valid ? v[q].w & 0xFFFFu : 0u;
    }
    uint32_t pr[4];
    float csum = 0.0f, xsum = 0.0f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const float sc = w4_pair_scale(p);
        const uint32_t ha = f2h(h2f(hv[p]) * sc), hb = f2h(h2f(hv[4 + p]) * sc);
        pr[p] = ha | (hb << 16);
        csum += h2f(ha) + h2f(hb);
        xsum += h2f(hv[p]) + h2f(hv[4 + p]);
    }
    csum = group_sum<4>(csum);
    xsum = group_sum<4>(xsum);
    if (valid) {
        const int ul = w >> 2, wi = w & 3;
        hs[wi * HS + ul] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        if (wi == 0)
            cx[ul] = make_float2(1024.0f * csum, xsum);
    }
}

// Loads of one gate/up wave-item: 8 rows from row0 (rows at or past row_end
// belong to another workgroup and are computed but never stored), 8 lanes
// per row.  Metadata of the 8 rows is contiguous per matrix; a 16-byte chunk
// whose row lies past the matrix is read from the item's first chunk instead.
template <int JG, int KM>
__device__ __forceinline__ void sk_gu_load(FGuItem<1, 8, JG, KM>& it, const StackLayer& w, int row0,
                                           int row_end, int f, int d, int g, int r, int lane) {
    const int s = lane & 7, U = d / 64, ng = d / g, chunks = 2 * ng;
    it.row0 = row0;
    it.row = row0 + (lane >> 3);
    it.ok = it.row < row_end;
    const long rowc = it.ok ? it.row : row0;
    const uint4* mg4 = reinterpret_cast<const uint4*>(w.mg);
    const uint4* mu4 = reinterpret_cast<const uint4*>(w.mu);
    const long mbase = (long)row0 * ng / 4;
#pragma unroll
    for (int k = 0; k < KM; ++k) {
        const int c = lane + 64 * k;
        const bool up = c >= chunks && c < 2 * chunks;
        const int cc = c < chunks ? c : (up ? c - chunks : 0);
        const bool inside = row0 + (4 * cc) / ng < f;
        it.meta[k] = load_stream((up ? mu4 : mg4) + mbase + (inside ? cc : 0));
    }
    const uint4* cg = reinterpret_cast<const uint4*>(w.cg) + rowc * U + s;
    const uint4* cu = reinterpret_cast<const uint4*>(w.cu) + rowc * U + s;
#pragma unroll
    for (int i = 0; i < JG; ++i) {          // U == 8 * JG: every slot is inside the row
        it.qg[i] = load_stream(cg + 8 * i);
        it.qu[i] = load_stream(cu + 8 * i);
    }
    // LoRA-B rows of the item, B_g then B_u: each matrix's 8 rows are r
    // contiguous 16-byte chunks, and lane c < 2r loads chunk c with one
    // branch-free load (a chunk past the matrix, and every lane at rank 0,
    // re-reads a valid chunk).  sk_gu_finish parks them in LDS.  Loads of
    // different widths under a rank-dependent branch would make the compiler
    // wait for every outstanding load where the branches merge, which turns
    // the next layer's prefetch into a synchronous load.
    {
        const int c = lane < 2 * r ? lane : 0;
        const bool up = c >= r && r > 0;
        const int cc = up ? c - r : c;
        const bool in = r > 0 && row0 + (8 * cc) / r < f;
        const uint4* base = r > 0 ? reinterpret_cast<const uint4*>(up ? w.Bu : w.Bg) + (long)row0 * r / 8
                                  : reinterpret_cast<const uint4*>(w.cg);
        const uint4 b = load_stream(base + (in ? cc : 0));
        it.bg[0] = b.x; it.bg[1] = b.y; it.bu[0] = b.z; it.bu[1] = b.w;
    }
    it.G[0] = it.U[0] = 0.0f;
}

// Gate/up dot products of one wave-item over the staged x' (one token, 8
// lanes per row, U == 8 * JG units): slot i of lane s is unit s + 8 i, its
// eight x' chunks read just before its arithmetic.  The per-group
// (scale, zero) words come from the wave's metadata area in LDS.
template <int JG, int KM>
__device__ __forceinline__ void sk_gu_accumulate(FGuItem<1, 8, JG, KM>& it, const uint4* xs,
                                                 const float2* cx, int g, const uint32_t* wmeta,
                                                 int lane) {
    constexpr int XS = 8 * JG;
    const uint32_t mv = magic_vgpr();
    const int s = lane & 7, r = lane >> 3;
    const int ng = XS * 64 / g, gsh = g == 128 ? 1 : 0;
    const uint4* xl = xs + s;
    const float2* cl = cx + s;
    const uint32_t* mgl = wmeta + r * ng + (s >> gsh);
    const uint32_t* mul = wmeta + (8 + r) * ng + (s >> gsh);
#pragma unroll
    for (int i = 0; i < JG; ++i) {
        uint4 xv[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) xv[c] = xl[c * XS + 8 * i];
        uint32_t wg[4] = {it.qg[i].x, it.qg[i].y, it.qg[i].z, it.qg[i].w};
        uint32_t wu[4] = {it.qu[i].x, it.qu[i].y, it.qu[i].z, it.qu[i].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            pin(wg[q]);
            pin(wu[q]);
        }
        float ag = 0.0f, au = 0.0f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t eg[8], eu[8];
            extract_w2(wg[q], eg, mv);
            extract_w2(wu[q], eu, mv);
            const uint32_t xp[8] = {xv[2 * q].x, xv[2 * q].y, xv[2 * q].z, xv[2 * q].w,
                                    xv[2 * q + 1].x, xv[2 * q + 1].y, xv[2 * q + 1].z, xv[2 * q + 1].w};
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                ag = dot2(eg[p], xp[p], ag);
                au = dot2(eu[p], xp[p], au);
            }
        }
        const int gi = (8 * i) >> gsh;
        const uint32_t mgi = mgl[gi], mui = mul[gi];
        const float2 k = cl[8 * i];
        it.G[0] += h2f(mgi & 0xFFFFu) * (ag - k.x - h2f(mgi >> 16) * k.y);
        it.U[0] += h2f(mui & 0xFFFFu) * (au - k.x - h2f(mui >> 16) * k.y);
    }
}

// LoRA-B on the lane's ranks (t unscaled: A x; the item's B rows go through
// the wave's LDS area wb, 32 r bytes), the row reduction over 8 lanes, the norm's 1/rms (G and U are linear in the block input x * inv)
// and h = SiLU(G) * U, published as tagged words to the XCD-local h buffer.
template <int JG, int KM>
__device__ __forceinline__ void sk_gu_finish(FGuItem<1, 8, JG, KM>& it, const float* ts, int r,
                                             float ls, uint32_t* hb, uint32_t tag, int lane, uint4* wb) {
    const int s = lane & 7;
    const float inv = ts[2 * r];           // 1 / rms of the stream: the block input is x * inv
    float G = it.G[0], U = it.U[0];
    if (r > 0) {
        // the item's LoRA-B rows into the wave's LDS area: [B_g rows | B_u rows], r halves per row
        if (lane < 2 * r)
            wb[lane] = make_uint4(it.bg[0], it.bg[1], it.bu[0], it.bu[1]);
        const uint16_t* bh = reinterpret_cast<const uint16_t*>(wb) + (lane >> 3) * r;
        const int CPL = r / 8;
        float lg = 0.0f, lu = 0.0f;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            if (c < CPL) {
                const int rc = s * CPL + c;
                lg += h2f(bh[rc]) * ts[rc];
                lu += h2f(bh[8 * r + rc]) * ts[r + rc];
            }
        }
        G += ls * lg;
        U += ls * lu;
    }
    // everything above is linear in the input: scale by 1/rms once per row
    G = group_sum<8>(G) * inv;
    U = group_sum<8>(U) * inv;
    if (it.ok && s == 0) {
        const float hv = G / (1.0f + __expf(-G)) * U;
        st_intra32(hb + it.row, f2h(hv) | (tag << 16));
    }
}

// One down wave-item: 8 output rows of D_j, 8 lanes per row; lane s owns the
// 32-code units s, s+8, ... of this XCD's column slice (UF units).  Each
// unit's (scale | zero) word is loaded with it (groups need not align with
// the slice).
template <int JD>
struct SkDn {
    uint4 q[JD];
    uint32_t mt[JD];
};

template <int JD>
__device__ __forceinline__ void sk_dn_load(SkDn<JD>& it, const StackLayer& w, int o, int xcc, int f,
                                           int g, int lane) {
    const int s = lane & 7, FX = f / SX, UF = FX / 32, Uf = f / 32, ngd = f / g;
    const uint4* cd = reinterpret_cast<const uint4*>(w.cd) + (long)o * Uf + xcc * UF;
    const uint32_t* md = w.md + (long)o * ngd;
#pragma unroll
    for (int i = 0; i < JD; ++i) {
        // only the last slot can run past the slice: it re-reads the slice's
        // last unit, and its contribution is dropped
        const int u = i + 1 < JD ? s + 8 * i : (s + 8 * i < UF ? s + 8 * i : UF - 1);
        it.q[i] = load_stream(cd + u);
        it.mt[i] = load_stream(md + (xcc * FX + 32 * u) / g);
    }
}

template <int JD>
__device__ __forceinline__ float sk_dn_compute(SkDn<JD>& it, const uint4* hs, const float2* hcx,
                                               int UF, int lane) {
    constexpr int HS = 8 * JD;
    const uint32_t mv = magic_vgpr();
    const int s = lane & 7;
    const uint4* hl = hs + s;
    const float2* cl = hcx + s;
    float Y = 0.0f;
#pragma unroll
    for (int i = 0; i < JD; ++i) {
        uint32_t wv[4] = {it.q[i].x, it.q[i].y, it.q[i].z, it.q[i].w};
        uint32_t mti = it.mt[i];
#pragma unroll
        for (int q = 0; q < 4; ++q) pin(wv[q]);
        pin(mti);
        float acc = 0.0f;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            uint32_t e[4];
            extract_w4(wv[q], e, mv);
            const uint4 p = hl[q * HS + 8 * i];
            acc = dot2(e[0], p.x, acc);
            acc = dot2(e[1], p.y, acc);
            acc = dot2(e[2], p.z, acc);
            acc = dot2(e[3], p.w, acc);
        }
        const float2 k = cl[8 * i];
        const float c = h2f(mti & 0xFFFFu) * (acc - k.x - h2f(mti >> 16) * k.y);
        if (i + 1 < JD || s + 8 * i < UF)
            Y += c;
    }
    return group_sum<8>(Y);
}

// Layer i's descriptor, read in place from the kernel-argument segment (the
// argument block starts with the layer array): indexing the by-value
// argument with a run-time layer index would copy the whole block to scratch.
template <class Args>
__device__ __forceinline__ StackLayer sk_layer(const Args __attribute__((address_space(4)))* ka, int i) {
    StackLayer w;
    w.cg = ka->lay[i].cg; w.mg = ka->lay[i].mg; w.cu = ka->lay[i].cu; w.mu = ka->lay[i].mu;
    w.cd = ka->lay[i].cd; w.md = ka->lay[i].md; w.Bg = ka->lay[i].Bg; w.Bu = ka->lay[i].Bu;
    w.Ag = ka->lay[i].Ag; w.Au = ka->lay[i].Au; w.lora_scale = ka->lay[i].lora_scale;
    return w;
}

}  // namespace

}  // namespace qmlp

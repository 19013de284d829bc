// Streamed decode path for a batch of independent blocks at one token
// (binary16), gfx950: two persistent launches.
//
//   gate/up launch:  t_l = [A_g; A_u] x_l, then
//                    h_l = SiLU(W2gate x_l + s B_g t_g) * (W2up x_l + s B_u t_u)
//                    for every block l of the batch (Sec. 3.1 Eq. (1),
//                    Sec. 3.3, Sec. 4.2);
//   down launch:     y_l = W4down h_l (Sec. 3.3).
//
// Decode is bound by loading weights (Sec. 1, Sec. 3.3).  The blocks of a
// batch do not depend on each other, so every workgroup owns one contiguous
// range of the batch's rows (flattened over blocks) and streams it, and the
// activation of the few blocks a range touches (x for gate/up, h for down)
// is staged in LDS once per launch.  The one hand-off inside a launch is t:
// each gate/up workgroup also computes a share of the batch's LoRA-A rows
// (one per wave, its loads issued ahead of the weights) and publishes them
// as tagged words, then reads the t of its own range's blocks before its
// staging barrier (the workgroups, one per compute unit, are all resident;
// the wait is bounded).  Each wave walks its share of the range with two
// register sets: the loads of its next step go out before the current
// step's arithmetic, in straight-line code with exact unit counts (the
// prefetch of a wave's last step re-reads a valid address and is dropped),
// so the compiler's wait counts stay partial and the load stream does not
// stop for arithmetic.
//
// Work items.  gate/up: 8 rows of gate and up, 8 lanes per row, lane s owns
// the 16-byte units s, s + 8, ... of its row (a row of d 2-bit codes is
// UG = d/64 units; JC of them per lane per step, NCH steps per row).  down:
// one row per wave, 64 lanes, lane s owns units s, s + 64, ... (f/32 units,
// padded to UD = 64 JD in LDS with zeros).
//
// Dequantization.  A code field OR-ed into the fraction of binary16 1024.0
// reads 1024 + q 2^j (j = its bit position inside the fraction), so
// v_dot2_f32_f16 of such a pair with an activation pair pre-scaled by 2^-j
// gives q x + 1024 x'; the per-unit sums C = 1024 sum x' and X = sum x,
// staged (negated) with the activation, remove the offset and the zero
// point: each unit's accumulator starts at -(C + z X) and
// sum s (q - z) x = s acc.  Fields are used where they sit in the
// code word, so a word needs one shift: at 2 bits the codes of each half at
// bits 0-9 read in place (positions 0, 2, 4, 6, 8) and the word shifted
// right by 6 brings the other three to positions 4, 6, 8; at 4 bits codes 0
// and 1 of each half read at positions 0 and 4, and the word shifted right
// by 8 brings codes 2 and 3 there.  The staged activation is chunk-major
// ([chunk][unit]), so the eight lanes of a row read consecutive 16-byte
// units (no bank conflicts) and every LDS read of a step is one base
// register plus an immediate offset.
#include "decode_common.h"
#include "decode_launch.h"

namespace qmlp {

namespace {

constexpr int kStreamSpan = 3;          // blocks one workgroup's range may touch
// Control words of the batch workspace (uint32 indices, each on its own
// 128-byte line): the call counter that tags t, sticky error bits.
constexpr int kStreamCtlEpoch = 0, kStreamCtlErr = 160;
constexpr unsigned kStreamSpinLimit = 1u << 18;

// The kernel's BatchArgs read in place from the kernel-argument segment, so
// indexing the descriptor table with a (wave-uniform) block index compiles to
// scalar loads instead of a private copy of the table.
typedef const BatchArgs __attribute__((address_space(4))) KBatch;
__device__ __forceinline__ KBatch* kbatch() { return (KBatch*)__builtin_amdgcn_kernarg_segment_ptr(); }

// Workgroup w's share [lo, hi) of n work items split over G workgroups.
__device__ __forceinline__ void wg_share(int n, int G, int w, int& lo, int& hi) {
    lo = (int)((long)w * n / G);
    hi = (int)((long)(w + 1) * n / G);
}

// A wave's walk over items item0, item0 + NW, ... of rows-per-item RPI in a
// batch of blocks of `per` rows: block l and first row n of the current item,
// advanced without a division.
struct Walk {
    int l, n;
    __device__ __forceinline__ void start(int item0, int rpi, int per) {
        l = item0 * rpi / per;
        n = item0 * rpi - l * per;
    }
    __device__ __forceinline__ void next(int stride_rows, int per) {    // stride_rows < per
        n += stride_rows;
        if (n >= per) {
            n -= per;
            ++l;
        }
    }
};

// ---------------------------------------------------------------- gate/up
// Staging word wi of one block's x (16 codes: word wi & 3 of unit wi >> 2)
// into x' chunks 2w, 2w + 1 of the unit (chunk-major, UG units per chunk)
// and the unit's (C, X).  The four words of a unit sit on four consecutive
// lanes; every lane of the wave calls this (shuffles); live = false stores
// nothing.
template <int UG>
__device__ __forceinline__ void gu_stage_word(uint4* xs, float2* cx, int wi, bool live, const XWord& v) {
    const int u = wi >> 2, w = wi & 3;
    const uint32_t xl[4] = {v.lo.x, v.lo.y, v.lo.z, v.lo.w};
    const uint32_t xh[4] = {v.hi.x, v.hi.y, v.hi.z, v.hi.w};
    uint32_t pr[8];
    float csum = 0.0f, xsum = 0.0f;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        const uint32_t a16 = (xl[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;     // x[p]
        const uint32_t b16 = (xh[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;     // x[8 + p]
        const float sc = w2_s1_scale(p);
        const uint32_t ha = f2h(h2f(a16) * sc), hb = f2h(h2f(b16) * sc);
        pr[p] = ha | (hb << 16);
        csum += h2f(ha) + h2f(hb);
        xsum += h2f(a16) + h2f(b16);
    }
    csum = group_sum<4>(csum);
    xsum = group_sum<4>(xsum);
    if (live) {
        xs[(2 * w) * UG + u] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        xs[(2 * w + 1) * UG + u] = make_uint4(pr[4], pr[5], pr[6], pr[7]);
        if (w == 0)
            cx[u] = make_float2(-1024.0f * csum, -xsum);          // (-C, -X)
    }
}

template <int JC>
struct GuBuf {
    uint4 qg[JC], qu[JC];
    uint32_t mg[JC], mu[JC];
    uint32_t bg[2], bu[2];      // LoRA-B: this lane's r/8 ranks of its row (raw binary16)
};

// Loads of step c of the item whose first row is row n of block l (lane:
// row n + lane/8).  Always issued, from valid addresses: a prefetch past a
// wave's last step (dummy) reads the batch's x instead, which the staging
// has just brought into the caches (every offset below stays inside the
// first 2d bytes of x).
template <int JC, int NCH, int R, int GSH>
__device__ __forceinline__ void gu_load(GuBuf<JC>& q, int l, int n, int c, bool dummy, const uint16_t* x,
                                        int lane) {
    constexpr int UG = 8 * JC * NCH;
    constexpr int NG = UG >> GSH;                        // groups per row (64 << GSH codes each)
    KBatch* kb = kbatch();
    const int row = (dummy ? 0 : n) + (lane >> 3), s = lane & 7;
    const void* pcg = dummy ? (const void*)x : (const void*)kb->lay[l].cg;
    const void* pcu = dummy ? (const void*)x : (const void*)kb->lay[l].cu;
    const void* pmg = dummy ? (const void*)x : (const void*)kb->lay[l].mg;
    const void* pmu = dummy ? (const void*)x : (const void*)kb->lay[l].mu;
    const uint4* cg = reinterpret_cast<const uint4*>(pcg) + row * UG + s + 8 * JC * c;
    const uint4* cu = reinterpret_cast<const uint4*>(pcu) + row * UG + s + 8 * JC * c;
    // unit s + 8 i lies in group (s >> GSH) + (8 >> GSH) i
    const uint32_t* mg = reinterpret_cast<const uint32_t*>(pmg) + row * NG + (s >> GSH) + (8 >> GSH) * JC * c;
    const uint32_t* mu = reinterpret_cast<const uint32_t*>(pmu) + row * NG + (s >> GSH) + (8 >> GSH) * JC * c;
#pragma unroll
    for (int j = 0; j < JC; ++j) {
        q.qg[j] = load_stream(cg + 8 * j);
        q.qu[j] = load_stream(cu + 8 * j);
        q.mg[j] = load_stream(mg + (8 >> GSH) * j);
        q.mu[j] = load_stream(mu + (8 >> GSH) * j);
    }
    const uint16_t* Bg = dummy ? x : kb->lay[l].Bg;
    const uint16_t* Bu = dummy ? x : kb->lay[l].Bu;
    if constexpr (R == 8) {
        q.bg[0] = Bg[row * R + s];
        q.bu[0] = Bu[row * R + s];
    } else if constexpr (R == 16) {
        q.bg[0] = reinterpret_cast<const uint32_t*>(Bg)[row * (R / 2) + s];
        q.bu[0] = reinterpret_cast<const uint32_t*>(Bu)[row * (R / 2) + s];
    } else if constexpr (R == 32) {
        const uint2 vg = reinterpret_cast<const uint2*>(Bg)[row * (R / 4) + s];
        const uint2 vu = reinterpret_cast<const uint2*>(Bu)[row * (R / 4) + s];
        q.bg[0] = vg.x; q.bg[1] = vg.y; q.bu[0] = vu.x; q.bu[1] = vu.y;
    }
}

// Arithmetic of step c into the lane's row sums G, U.  xl = the staged x' of
// the row's block + this lane's unit (s); cl likewise for (C, X).
template <int JC, int NCH>
__device__ __forceinline__ void gu_dot(GuBuf<JC>& q, const uint4* xl, const float2* cl, int c, float& G,
                                       float& Uv) {
    constexpr int UG = 8 * JC * NCH;
    const uint32_t mv = magic_vgpr();
#pragma unroll
    for (int j = 0; j < JC; ++j) {
        const int uo = 8 * (JC * c + j);                 // unit offset of slot j (compile time)
        uint32_t wg[4] = {q.qg[j].x, q.qg[j].y, q.qg[j].z, q.qg[j].w};
        uint32_t wu[4] = {q.qu[j].x, q.qu[j].y, q.qu[j].z, q.qu[j].w};
        uint32_t mgi = q.mg[j], mui = q.mu[j];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            pin(wg[w]);
            pin(wu[w]);
        }
        pin(mgi);
        pin(mui);
        // the accumulators start at -(C + z X) (cl holds -C, -X): the unit's
        // sum is then s * acc
        const float2 k = cl[uo];
        float ag = h2f(mgi >> 16) * k.y + k.x;
        float au = h2f(mui >> 16) * k.y + k.x;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            uint32_t eg[8], eu[8];
            extract_w2_s1(wg[w], eg, mv);
            extract_w2_s1(wu[w], eu, mv);
            const uint4 p0 = xl[(2 * w) * UG + uo];
            const uint4 p1 = xl[(2 * w + 1) * UG + uo];
            const uint32_t xp[8] = {p0.x, p0.y, p0.z, p0.w, p1.x, p1.y, p1.z, p1.w};
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                ag = dot2(eg[p], xp[p], ag);
                au = dot2(eu[p], xp[p], au);
            }
        }
        G += h2f(mgi & 0xFFFFu) * ag;
        Uv += h2f(mui & 0xFFFFu) * au;
    }
}

// LoRA-B, the row reduction over 8 lanes and SiLU(G) * U into the LDS copy
// of the range's h (hs: this item's 8 values).  The loop stores nothing to
// memory: a store counts in the same in-order counter as the loads, so a
// store inside the loop makes the next prefetch wait for every earlier load.
template <int JC, int R>
__device__ __forceinline__ void gu_finish(GuBuf<JC>& q, const float* ts, int l, uint16_t* hs, int lane,
                                          float G, float Uv) {
    const int s = lane & 7;
    if constexpr (R > 0) {
        constexpr int CPL = R / 8;               // ranks per lane
        float lg = 0.0f, lu = 0.0f;
        uint32_t bgv[2] = {q.bg[0], q.bg[1]}, buv[2] = {q.bu[0], q.bu[1]};
        pin(bgv[0]); pin(bgv[1]); pin(buv[0]); pin(buv[1]);
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const uint32_t hg = (bgv[c >> 1] >> (16 * (c & 1))) & 0xFFFFu;
            const uint32_t hu = (buv[c >> 1] >> (16 * (c & 1))) & 0xFFFFu;
            lg += h2f(hg) * ts[s * CPL + c];
            lu += h2f(hu) * ts[R + s * CPL + c];
        }
        const float sl = kbatch()->lay[l].lora_scale;
        G += sl * lg;
        Uv += sl * lu;
    }
    G = group_sum<8>(G);
    Uv = group_sum<8>(Uv);
    if (s == 0)
        hs[lane >> 3] = (uint16_t)f2h(G / (1.0f + __expf(-G)) * Uv);
}

template <int JC, int NCH, int R, int GSH, int NW>
__global__ void __launch_bounds__(NW * 64) gu_stream_kernel(BatchArgs b, int nb, int span,
                                                            unsigned long long* t64, unsigned* ctl) {
    static_assert(NCH == 1 || NCH == 2, "one or two steps per row");
    constexpr int NT = NW * 64, UG = 8 * JC * NCH;
    const int f = b.f;
    extern __shared__ uint4 smem[];
    uint4* xs = smem;                                                   // [span][8][UG]
    float2* cx = reinterpret_cast<float2*>(smem + span * 8 * UG);       // [span][UG]
    float* ts = reinterpret_cast<float*>(cx + span * UG);               // [span][2R]
    uint16_t* hout = reinterpret_cast<uint16_t*>(ts + span * 2 * R);    // [8 (i1 - i0)]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // LoRA-A: the workgroup's share [c0, c1) of the rows of the batch's
    // [nb][2R] t, row c0 + w on wave w, whose loads go out first and whose
    // product is published as a tagged word (fp32 | tag << 32, tag = the
    // call counter plus one) after the staging (rows past the waves follow
    // one per wave at a time); every workgroup then reads the t of its range's blocks,
    // which other workgroups of this launch (all resident: one per compute
    // unit) publish.
    constexpr int KA = JC * NCH;                 // 8-element chunks of a row per lane (d / 512)
    int c0 = 0, c1 = 0;
    if constexpr (R > 0)
        wg_share(nb * 2 * R, gridDim.x, blockIdx.x, c0, c1);
    const int lc = c0 + wave;
    const bool lw = R > 0 && lc < c1;
    uint4 la[R > 0 ? KA : 1], lx[R > 0 ? KA : 1];
    if constexpr (R > 0) {
        if (lw) {
            KBatch* kb = kbatch();
            const int l = lc / (2 * R), row = lc - l * 2 * R;
            const uint16_t* arow = row < R ? kb->lay[l].Ag + (long)row * b.d : kb->lay[l].Au + (long)(row - R) * b.d;
            const uint16_t* xrow = b.x + (long)l * b.d;
#pragma unroll
            for (int k = 0; k < KA; ++k) {
                la[k] = *reinterpret_cast<const uint4*>(arow + (lane + 64 * k) * 8);
                lx[k] = *reinterpret_cast<const uint4*>(xrow + (lane + 64 * k) * 8);
            }
        }
    }
    unsigned epoch = 0;
    if constexpr (R > 0)
        epoch = __hip_atomic_load(ctl + kStreamCtlEpoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    int i0, i1;
    wg_share(nb * (f / 8), gridDim.x, blockIdx.x, i0, i1);
    const int l0 = i0 * 8 / f;
    const int nbk = i1 > i0 ? (i1 * 8 - 1) / f - l0 + 1 : 0;           // <= span (host)

    // this wave's items: i0 + wave, i0 + wave + NW, ...; NCH steps each
    const int first = i0 + wave;
    const int nk = first < i1 ? (i1 - first + NW - 1) / NW : 0;
    const int nsteps = nk * NCH;

    // x of the range's blocks: loaded first (loads retire in order), then the
    // first step's weights, then the conversion into x'.
    constexpr int XW = (kStreamSpan * UG * 4 + NT - 1) / NT;    // staging words per thread
    XWord xv[XW];
    const int words = nbk * UG * 4;
#pragma unroll
    for (int k = 0; k < XW; ++k) {
        const int idx = tid + NT * k;
        const int wi = idx < words ? idx : 0;
        const uint4* src = reinterpret_cast<const uint4*>(b.x + (long)l0 * b.d) + 2 * wi;
        xv[k] = XWord{src[0], src[1]};
    }
    __builtin_amdgcn_sched_barrier(0);
    Walk ld, cp;                      // the next step to load / to compute
    int ldc = 0;
    GuBuf<JC> A, B;
    if (nsteps > 0) {
        ld.start(first, 8, f);
        cp = ld;
        gu_load<JC, NCH, R, GSH>(A, ld.l, ld.n, 0, false, b.x, lane);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < XW; ++k) {
        const int idx = tid + NT * k;
        const int bb = idx < words ? idx / (UG * 4) : 0;
        const int wi = idx < words ? idx - bb * UG * 4 : 0;
        gu_stage_word<UG>(xs + bb * 8 * UG, cx + bb * UG, wi, idx < words, xv[k]);
    }
    if constexpr (R > 0) {
        const unsigned long long tag = epoch % 0xFFFFFFFFu + 1u;
        if (lw) {
            float acc = 0.0f;
#pragma unroll
            for (int k = 0; k < KA; ++k) {
                acc = dot2(la[k].x, lx[k].x, acc);
                acc = dot2(la[k].y, lx[k].y, acc);
                acc = dot2(la[k].z, lx[k].z, acc);
                acc = dot2(la[k].w, lx[k].w, acc);
            }
            acc = group_sum<64>(acc);
            if (lane == 0)
                __hip_atomic_store(t64 + lc, (unsigned long long)__float_as_uint(acc) | (tag << 32),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        // a share longer than the waves (many blocks at rank 32): the rest,
        // one row per wave at a time
        for (int c = lc + NW; c < c1; c += NW) {
            KBatch* kb = kbatch();
            const int l = c / (2 * R), row = c - l * 2 * R;
            const uint16_t* arow = row < R ? kb->lay[l].Ag + (long)row * b.d : kb->lay[l].Au + (long)(row - R) * b.d;
            const float v = lora_a_dot<KA>(arow, b.x + (long)l * b.d, b.d, lane);
            if (lane == 0)
                __hip_atomic_store(t64 + c, (unsigned long long)__float_as_uint(v) | (tag << 32),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    if constexpr (R > 0) {
        // t of the range's blocks: re-read until a word shows this call's tag
        // (bounded: after kStreamSpinLimit polls the word is taken as it is
        // and error bit 1 is set)
        const unsigned tag = epoch % 0xFFFFFFFFu + 1u;
        for (int k = tid; k < nbk * 2 * R; k += NT) {
            const unsigned long long* p = t64 + (long)l0 * 2 * R + k;
            unsigned long long v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (unsigned n = 0; (unsigned)(v >> 32) != tag && n < kStreamSpinLimit; ++n) {
                __builtin_amdgcn_s_sleep(2);
                v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            if ((unsigned)(v >> 32) != tag)
                __hip_atomic_fetch_or(ctl + kStreamCtlErr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            ts[k] = __uint_as_float((uint32_t)v);
        }
    }
    __syncthreads();

    // step bookkeeping: load position advances after each issued load while
    // steps remain (the last step's prefetch repeats the last load)
    int left = nsteps - 1;            // loads still to issue after the first
    auto advance_load = [&]() {       // false: the next load is a dummy
        if (left > 0) {
            --left;
            if (++ldc == NCH) {
                ldc = 0;
                ld.next(8 * NW, f);
            }
            return true;
        }
        return false;
    };
    float G = 0.0f, Uv = 0.0f;
    int ci = first - i0;                 // the computed item's index inside the range
    auto run = [&](GuBuf<JC>& q, int c) {
        const int bb = cp.l - l0;
        const int s = lane & 7;
        gu_dot<JC, NCH>(q, xs + bb * 8 * UG + s, cx + bb * UG + s, c, G, Uv);
        if (c == NCH - 1) {
            gu_finish<JC, R>(q, ts + bb * 2 * R, cp.l, hout + 8 * ci, lane, G, Uv);
            G = Uv = 0.0f;
            cp.next(8 * NW, f);
            ci += NW;
        }
    };
    // one back edge and no exit in the middle: both halves always issue
    // their loads, the second half skips its arithmetic past the last step
    for (int st = 0; st < nsteps; st += 2) {
        bool real = advance_load();
        gu_load<JC, NCH, R, GSH>(B, ld.l, ld.n, NCH - 1, !real, b.x, lane);
        run(A, 0);
        real = advance_load();
        gu_load<JC, NCH, R, GSH>(A, ld.l, ld.n, 0, !real, b.x, lane);
        if (st + 1 < nsteps)
            run(B, NCH - 1);
    }
    // the range's h: 8 (i1 - i0) contiguous values of the batch's flattened
    // [nb][f], written as 16-byte words (one item per thread and round)
    __syncthreads();
    uint4* hdst = reinterpret_cast<uint4*>(b.h) + i0;
    const uint4* hsrc = reinterpret_cast<const uint4*>(hout);
    for (int k = tid; k < i1 - i0; k += NT)
        hdst[k] = hsrc[k];
}

// ---------------------------------------------------------------- down
// Staging word wi of one block's h (8 codes: word wi & 3 of unit wi >> 2)
// into h' chunk w of the unit (chunk-major, UD units per chunk) and the
// unit's (C, X); live = false stores nothing.
template <int UD>
__device__ __forceinline__ void dn_stage_word(uint4* hs, float2* cx, int wi, bool live, uint4 v) {
    const int u = wi >> 2, w = wi & 3;
    const uint32_t hl[4] = {v.x, v.y, v.z, v.w};
    uint32_t pr[4];
    float csum = 0.0f, xsum = 0.0f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t a16 = (hl[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;         // h[p]
        const uint32_t b16 = (hl[2 + (p >> 1)] >> (16 * (p & 1))) & 0xFFFFu;   // h[4 + p]
        const float sc = w4_s1_scale(p);
        const uint32_t ha = f2h(h2f(a16) * sc), hb = f2h(h2f(b16) * sc);
        pr[p] = ha | (hb << 16);
        csum += h2f(ha) + h2f(hb);
        xsum += h2f(a16) + h2f(b16);
    }
    csum = group_sum<4>(csum);
    xsum = group_sum<4>(xsum);
    if (live) {
        hs[w * UD + u] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        if (w == 0)
            cx[u] = make_float2(-1024.0f * csum, -xsum);          // (-C, -X)
    }
}

template <int JD>
struct DnBuf {
    uint4 q[JD];
    uint32_t m[JD];
};

// Loads of row o of block l; a dummy prefetch (past a wave's last row)
// reads the batch's h instead (offsets below f/2 bytes), which the staging
// has just brought into the caches.
template <int JD>
__device__ __forceinline__ void dn_load(DnBuf<JD>& q, int l, int o, int U, int ng, int gsh, bool dummy,
                                        const uint16_t* h, int lane) {
    KBatch* kb = kbatch();
    const uint4* cd = dummy ? reinterpret_cast<const uint4*>(h)
                            : reinterpret_cast<const uint4*>(kb->lay[l].cd) + (long)o * U;
    const uint32_t* md = dummy ? reinterpret_cast<const uint32_t*>(h) : kb->lay[l].md + (long)o * ng;
#pragma unroll
    for (int j = 0; j < JD; ++j) {
        const int u = lane + 64 * j;
        const int uu = u < U ? u : U - 1;            // padding slots re-read the last unit
        q.q[j] = load_stream(cd + uu);
        q.m[j] = load_stream(md + (uu >> gsh));
    }
}

// hl/cl: the staged h' and (C, X) of the row's block + this lane's unit.
// Padding units are staged as zeros, so they add nothing.
template <int JD>
__device__ __forceinline__ float dn_dot(DnBuf<JD>& q, const uint4* hl, const float2* cl) {
    constexpr int UD = 64 * JD;
    const uint32_t mv = magic_vgpr();
    float y = 0.0f;
#pragma unroll
    for (int j = 0; j < JD; ++j) {
        uint32_t wv[4] = {q.q[j].x, q.q[j].y, q.q[j].z, q.q[j].w};
        uint32_t mi = q.m[j];
#pragma unroll
        for (int w = 0; w < 4; ++w) pin(wv[w]);
        pin(mi);
        const float2 k = cl[64 * j];                     // (-C, -X)
        float acc = h2f(mi >> 16) * k.y + k.x;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            uint32_t e[4];
            extract_w4_s1(wv[w], e, mv);
            const uint4 p = hl[w * UD + 64 * j];
            acc = dot2(e[0], p.x, acc);
            acc = dot2(e[1], p.y, acc);
            acc = dot2(e[2], p.z, acc);
            acc = dot2(e[3], p.w, acc);
        }
        y += h2f(mi & 0xFFFFu) * acc;
    }
    return y;
}

template <int JD, int NW, int NBUF>
__global__ void __launch_bounds__(NW * 64) dn_stream_kernel(BatchArgs b, int nb, int span, unsigned* ctl) {
    static_assert(NBUF == 2 || NBUF == 3, "two or three register sets");
    constexpr int NT = NW * 64, UD = 64 * JD;
    const int d = b.d, f = b.f, U = f / 32, gsh = b.gd == 128 ? 2 : 1, ng = f / b.gd;
    extern __shared__ uint4 smem[];
    uint4* hs = smem;                                                   // [span][4][UD]
    float2* cx = reinterpret_cast<float2*>(smem + span * 4 * UD);       // [span][UD]
    uint16_t* yout = reinterpret_cast<uint16_t*>(cx + span * UD);       // [r1 - r0]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // one lane of the first workgroup advances the call counter (with
    // adapters): its load goes out first and the store comes at the end
    const bool leader = ctl && b.r > 0 && tid == 0 && blockIdx.x == 0;
    unsigned epoch = 0;
    if (leader)
        epoch = __hip_atomic_load(ctl + kStreamCtlEpoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    int r0, r1;
    wg_share(nb * d, gridDim.x, blockIdx.x, r0, r1);
    const int l0 = r0 / d;
    const int nbk = r1 > r0 ? (r1 - 1) / d - l0 + 1 : 0;

    const int first = r0 + wave;
    const int nk = first < r1 ? (r1 - first + NW - 1) / NW : 0;

    // staging words span the padded units (UD per block), those past U stage zeros
    constexpr int HW = (kStreamSpan * UD * 4 + NT - 1) / NT;
    uint4 hv[HW];
    const int words = nbk * UD * 4;
#pragma unroll
    for (int k = 0; k < HW; ++k) {
        const int idx = tid + NT * k;
        const int bb = idx < words ? idx / (UD * 4) : 0;
        const int wi = idx < words ? idx - bb * UD * 4 : 0;
        const int wc = wi < U * 4 ? wi : 0;
        hv[k] = reinterpret_cast<const uint4*>(b.h + (long)(l0 + bb) * f)[wc];
    }
    __builtin_amdgcn_sched_barrier(0);
    Walk ld, cp;
    DnBuf<JD> A, B, C;
    int left = nk - 1;
    auto advance_load = [&]() {       // false: the next load is a dummy
        if (left > 0) {
            --left;
            ld.next(NW, d);
            return true;
        }
        return false;
    };
    if (nk > 0) {
        ld.start(first, 1, d);
        cp = ld;
        dn_load<JD>(A, ld.l, ld.n, U, ng, gsh, false, b.h, lane);
        if constexpr (NBUF == 3) {
            const bool real = advance_load();
            dn_load<JD>(B, ld.l, ld.n, U, ng, gsh, !real, b.h, lane);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < HW; ++k) {
        const int idx = tid + NT * k;
        const int bb = idx < words ? idx / (UD * 4) : 0;
        const int wi = idx < words ? idx - bb * UD * 4 : 0;
        const bool data = idx < words && wi < U * 4;
        const uint4 v = data ? hv[k] : make_uint4(0u, 0u, 0u, 0u);
        dn_stage_word<UD>(hs + bb * 4 * UD, cx + bb * UD, wi, idx < words, v);
    }
    __syncthreads();

    // the loop stores its rows into LDS only (see gu_finish)
    int ci = first - r0;
    auto run = [&](DnBuf<JD>& q) {
        const int bb = cp.l - l0;
        const float v = group_sum<64>(dn_dot<JD>(q, hs + bb * 4 * UD + lane, cx + bb * UD + lane));
        if (lane == 0)
            yout[ci] = (uint16_t)f2h(v);
        cp.next(NW, d);
        ci += NW;
    };
    if constexpr (NBUF == 2) {
        for (int st = 0; st < nk; st += 2) {
            bool real = advance_load();
            dn_load<JD>(B, ld.l, ld.n, U, ng, gsh, !real, b.h, lane);
            run(A);
            real = advance_load();
            dn_load<JD>(A, ld.l, ld.n, U, ng, gsh, !real, b.h, lane);
            if (st + 1 < nk)
                run(B);
        }
    } else {
        for (int st = 0; st < nk; st += 3) {
            bool real = advance_load();
            dn_load<JD>(C, ld.l, ld.n, U, ng, gsh, !real, b.h, lane);
            run(A);
            real = advance_load();
            dn_load<JD>(A, ld.l, ld.n, U, ng, gsh, !real, b.h, lane);
            if (st + 1 < nk)
                run(B);
            real = advance_load();
            dn_load<JD>(B, ld.l, ld.n, U, ng, gsh, !real, b.h, lane);
            if (st + 2 < nk)
                run(C);
        }
    }
    // the range's y: r1 - r0 contiguous values of the batch's flattened [nb][d]
    __syncthreads();
    for (int k = tid; k < r1 - r0; k += NT)
        b.y[r0 + k] = yout[k];
    if (leader)
        __hip_atomic_store(ctl + kStreamCtlEpoch, epoch + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- host side
// Waves per workgroup (one workgroup per compute unit): gate/up with one
// step per row (<= 168 VGPRs) runs three waves per SIMD, with two steps per
// row two; down four.
template <int NCH>
constexpr int gu_waves() { return NCH == 1 ? 12 : 8; }
constexpr int kDnWaves = 16, kDnBufs = 2;

int stream_cu_count() {
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

// The most blocks any workgroup's share of n items (of `per` items per
// block) touches.
int max_span(long n, long per, int G) {
    int span = 0;
    for (int w = 0; w < G; ++w) {
        const long lo = (long)w * n / G, hi = (long)(w + 1) * n / G;
        if (hi > lo) {
            const int s = (int)((hi - 1) / per - lo / per + 1);
            span = s > span ? s : span;
        }
    }
    return span;
}

int gu_steps(int UG, int& jc) {             // NCH, or 0 if the width is not built
    if (UG % 8 != 0)
        return 0;
    const int jg = UG / 8;
    if (jg <= 5) { jc = jg; return 1; }
    if (jg % 2 == 0 && jg / 2 <= 5) { jc = jg / 2; return 2; }
    return 0;
}

int dn_slots(int f) { return (f / 32 + 63) / 64; }

size_t gu_lds(int span, int UG, int r, int nb, int f, int G) {
    const size_t items = ((size_t)nb * f / 8 + G - 1) / G;          // most items of one range
    return (size_t)span * (UG * 8 * 16 + UG * 8 + 2 * r * 4) + items * 16;
}
size_t dn_lds(int span, int UD, int nb, int d, int G) {
    const size_t rows = ((size_t)nb * d + G - 1) / G;
    return (size_t)span * UD * (4 * 16 + 8) + (rows * 2 + 15) / 16 * 16;
}
int gu_span(int nb, int f, int G) { return max_span((long)nb * f / 8, f / 8, G); }
int dn_span(int nb, int d, int G) { return max_span((long)nb * d, d, G); }
// One workgroup per compute unit, fewer when the batch has fewer items.
int gu_grid(int nb, int f) {
    const long n = (long)nb * f / 8, c = stream_cu_count();
    return (int)(n < c ? n : c);
}
int dn_grid(int nb, int d) {
    const long n = (long)nb * d, c = stream_cu_count();
    return (int)(n < c ? n : c);
}

}  // namespace

bool stream_supported(int M, int d, int f, int gg, int bg, int gd, int bd, int r, int nb) {
    if (M != 1 || bg != 2 || bd != 4 || (gg != 64 && gg != 128) || (gd != 64 && gd != 128))
        return false;
    if (r != 0 && r != 8 && r != 16 && r != 32)
        return false;
    if (nb < 1 || nb > kBatchMax || d % 512 != 0 || f % 128 != 0 || d > 4096 || dn_slots(f) > 6)
        return false;
    int jc = 0;
    if (!gu_steps(d / 64, jc))
        return false;
    if (stream_cu_count() <= 0)
        return false;
    const int sg = gu_span(nb, f, gu_grid(nb, f)), sd = dn_span(nb, d, dn_grid(nb, d));
    if (sg > kStreamSpan || sd > kStreamSpan)
        return false;
    return gu_lds(sg, d / 64, r, nb, f, gu_grid(nb, f)) <= 64 * 1024 &&
           dn_lds(sd, 64 * dn_slots(f), nb, d, dn_grid(nb, d)) <= 64 * 1024;
}

#define QMLP_GUS(JC_, NCH_, R_)                                                           \
    if (jc == JC_ && nch == NCH_ && r == R_) {                                            \
        constexpr int NW = gu_waves<NCH_>();                                              \
        if (b.gg == 128)                                                                  \
            gu_stream_kernel<JC_, NCH_, R_, 1, NW><<<G, NW * 64, lds, st>>>(b, nb, span, t64, ctl); \
        else                                                                              \
            gu_stream_kernel<JC_, NCH_, R_, 0, NW><<<G, NW * 64, lds, st>>>(b, nb, span, t64, ctl); \
        return hipGetLastError();                                                         \
    }
#define QMLP_GUS_R(JC_, NCH_) QMLP_GUS(JC_, NCH_, 0) QMLP_GUS(JC_, NCH_, 8) QMLP_GUS(JC_, NCH_, 16) \
    QMLP_GUS(JC_, NCH_, 32)

hipError_t launch_gateup_stream(const BatchArgs& b, int nb, unsigned long long* t64, unsigned* ctl,
                                hipStream_t st) {
    if (!stream_supported(b.M, b.d, b.f, b.gg, b.bg, b.gd, b.bd, b.r, nb) || (b.r > 0 && (!t64 || !ctl)))
        return hipErrorInvalidValue;
    const int G = gu_grid(nb, b.f), r = b.r;
    int jc = 0;
    const int nch = gu_steps(b.d / 64, jc);
    const int span = gu_span(nb, b.f, G);
    const size_t lds = gu_lds(span, b.d / 64, r, nb, b.f, G);
    QMLP_GUS_R(1, 1) QMLP_GUS_R(2, 1) QMLP_GUS_R(3, 1) QMLP_GUS_R(4, 1) QMLP_GUS_R(5, 1)
    QMLP_GUS_R(3, 2) QMLP_GUS_R(4, 2) QMLP_GUS_R(5, 2)
    return hipErrorInvalidValue;
}

#define QMLP_DNS(JD_)                                                                     \
    if (jd == JD_) {                                                                      \
        dn_stream_kernel<JD_, kDnWaves, kDnBufs><<<G, kDnWaves * 64, lds, st>>>(b, nb, span, ctl); \
        return hipGetLastError();                                                         \
    }

hipError_t launch_down_stream(const BatchArgs& b, int nb, unsigned* ctl, hipStream_t st) {
    if (!stream_supported(b.M, b.d, b.f, b.gg, b.bg, b.gd, b.bd, b.r, nb))
        return hipErrorInvalidValue;
    const int G = dn_grid(nb, b.d);
    const int jd = dn_slots(b.f);
    const int span = dn_span(nb, b.d, G);
    const size_t lds = dn_lds(span, 64 * jd, nb, b.d, G);
    QMLP_DNS(1) QMLP_DNS(2) QMLP_DNS(3) QMLP_DNS(4) QMLP_DNS(5) QMLP_DNS(6)
    return hipErrorInvalidValue;
}

}  // namespace qmlp

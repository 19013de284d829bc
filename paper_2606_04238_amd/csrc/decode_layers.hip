// L independent decode MLP blocks in one persistent launch (M = 1,
// binary16), gfx950.
//
// Each block is the W4/W2-GateUp MLP with Recover-LoRA adapters (Sec. 3.1
// Eq. (1), Sec. 3.3, Sec. 4.2) on its own input x_l:
//   G = W2gate x_l + s B_g (A_g x_l),  U = W2up x_l + s B_u (A_u x_l),
//   h = SiLU(G) * U,  y_l = W4down h.
// No block reads another block's output, so the launch runs them as a
// software pipeline: the work of one iteration is
//   * the gate/up rows of block i (h_i published inside the XCD),
//   * the partial down sums of block i-2 (published to the other XCDs),
// while the two polling waves stage block i+1's input and gather h_{i-1} of
// the XCD.  Every hand-off inside the loop is consumed one iteration after it
// was published, and one barrier per iteration separates producers and
// consumers of the LDS buffers (double-buffered by parity).  The eight
// cross-XCD partials of every block's y have a slot per block and are summed
// after the last iteration, so inside the loop no XCD waits for another.
// Decode is bound by loading weights (Sec. 3.3, Sec. 5): every register set
// of weights is requested well before its arithmetic (gate/up: right after
// the previous block's; down: double-buffered where the registers allow), so
// the stream never waits for a hand-off.
//
// Work split (8 XCDs x 32 compute units, one 768-thread workgroup each), per
// block as in the persistent stack kernel: XCD x owns the slice
// F_x = [x f/8, (x+1) f/8) of the intermediate dimension; its workgroup j
// computes gate/up rows F_x,j and the partial down product over F_x for the
// output rows D_j = [j d/32, (j+1) d/32).  Workgroup j of XCD x sums the
// eight partials of the rows D_j[x DJ/8, (x+1) DJ/8) (DJ = d/32) of every
// block in XCD order and writes them.  The LoRA-A products A x_l of all
// blocks (fp32) are computed once at the start, one dot product per polling
// wave, and read back as tagged words.
//
// Which compute wave takes which gate/up wave-item and which run of down
// wave-items is a host-side plan in the kernel arguments: waves w and w + 4
// share a SIMD, and the plan balances the dequant work of each SIMD.
//
// Tags: h words carry stag(step) in their high half and sit in slot
// step & 3 of a four-slot buffer, step = seq0 + 1 + l counted across
// launches; a workgroup overwrites slot s only after every workgroup of its
// XCD has staged the h that was there (it has seen their h two steps later,
// published after their barrier that followed the staging), and clears its
// rows of all four slots when a launch starts.  The 64-bit words (LoRA-A
// products, down partials) carry a 32-bit tag of the step and have one slot
// per block.
#include <type_traits>

#include "stack_common.h"

namespace qmlp {

namespace {

// Control words (uint32 index into the control block).
constexpr int L_SEQ = 0, L_DONE = 32, L_ERR = 64, L_XC = 96;


constexpr int LCW = 10;                  // compute waves: gate/up waves first, then down waves
constexpr int LTHREADS = (LCW + SPW) * 64;
constexpr int LGU_MAX = 6;               // gate/up waves (one wave-item each) at most

}  // namespace

constexpr int kLayersMaxLayers = 40;            // blocks per launch (kernel-argument block < 4 KB)

struct LayersArgs {
    StackLayer lay[kLayersMaxLayers];
    int L, d, f, g, r;
    const uint16_t* x;           // [L][d] inputs
    uint16_t* y;                 // [L][d] outputs
    unsigned long long* tb;      // [kLayersMaxLayers][2r] LoRA-A products, fp32 | tag << 32
    uint32_t* hb;                // [4][f] XCD-local h words, binary16 | tag << 16
    unsigned long long* pb;      // [kLayersMaxLayers][8][d] partial down sums, fp32 | tag << 32
    unsigned* ctl;
    int n_gu;                    // compute waves 0 .. n_gu-1 each run gate/up wave-item `wave`
    int dn_lo[LCW], dn_n[LCW];   // down wave-items [dn_lo, dn_lo + dn_n) of the other compute waves
    int o_xs, o_cx, o_t, o_hs, o_hcx, o_meta, meta_bytes;   // LDS byte offsets
    int o_dmeta;                 // LDS: down metadata areas, 512 B per (compute wave, item)
};

namespace {

typedef const LayersArgs __attribute__((address_space(4))) LKArgs;

struct SlLds {
    uint4* xs;          // [2][8 UG] x' of the activation (gate/up units), by block parity
    float2* cx;         // [2][UG] per unit (1024 sum x', sum x)
    float* ts;          // [2][2r + 1] A x (fp32), then 1 (no norm)
    uint4* hs;          // [2][4 HS] h' of this XCD's slice (down units)
    float2* hcx;        // [2][HS] per unit (1024 sum h', sum h)
    char* meta;         // per-wave gate/up metadata areas
    uint4* dmeta;       // down metadata: 32 16-byte chunks per (compute wave, item)
};

// Staging word w of block l's input: x[16w, 16w + 16) into the gate/up x'
// layout (pairs (x[16w+p], x[16w+8+p]) pre-scaled by their fraction
// position; chunk 2(w&3) holds pairs 0..3, chunk 2(w&3)+1 pairs 4..7 of unit
// w/4) and the unit sums.  The four words of a unit sit on four consecutive
// lanes.
template <int XS>
__device__ __forceinline__ void sl_stage_x(uint4* xs, float2* cx, const uint4 (&v)[2], bool valid, int w) {
    const uint32_t lo[8] = {v[0].x, v[0].y, v[0].z, v[0].w, v[1].x, v[1].y, v[1].z, v[1].w};
    uint32_t pr[8];
    float csum = 0.0f, xsum = 0.0f;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        // x[16w + p] is half p of the first 16 bytes, x[16w + 8 + p] of the second
        const uint32_t a = valid ? (lo[p >> 1] >> (16 * (p & 1))) & 0xFFFFu : 0u;
        const uint32_t b = valid ? (lo[4 + (p >> 1)] >> (16 * (p & 1))) & 0xFFFFu : 0u;
        const float sc = w2_pair_scale(p);
        const uint32_t ha = f2h(h2f(a) * sc), hb = f2h(h2f(b) * sc);
        pr[p] = ha | (hb << 16);
        csum += h2f(ha) + h2f(hb);
        xsum += h2f(a) + h2f(b);
    }
    csum = group_sum<4>(csum);
    xsum = group_sum<4>(xsum);
    if (valid) {
        const int ul = w >> 2, wi = w & 3;
        xs[(2 * wi) * XS + ul] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        xs[(2 * wi + 1) * XS + ul] = make_uint4(pr[4], pr[5], pr[6], pr[7]);
        if (wi == 0)
            cx[ul] = make_float2(1024.0f * csum, xsum);
    }
}

// Per-lane offsets of a gate/up wave-item's loads (the same for every block:
// only the base pointers change), in the order sk_gu_load issues them.
template <int KM>
struct SlGuAddr {
    long moff[KM];      // metadata chunk (16-byte units) and whether it is an up chunk
    bool mup[KM];
    long coff;          // codes of slot 0 (16-byte units); slot i at coff + 8 i
    long boff;          // LoRA-B chunk (16-byte units) and whether it is an up chunk
    bool bup;
};

template <int KM>
__device__ __forceinline__ SlGuAddr<KM> sl_gu_addr(int row0, int row_end, int f, int d, int g, int r, int lane) {
    SlGuAddr<KM> a;
    const int s = lane & 7, U = d / 64, ng = d / g, chunks = 2 * ng;
    const int row = row0 + (lane >> 3);
    const long rowc = row < row_end ? row : row0;
    const long mbase = (long)row0 * ng / 4;
#pragma unroll
    for (int k = 0; k < KM; ++k) {
        const int c = lane + 64 * k;
        const bool up = c >= chunks && c < 2 * chunks;
        const int cc = c < chunks ? c : (up ? c - chunks : 0);
        const bool inside = row0 + (4 * cc) / ng < f;
        a.moff[k] = mbase + (inside ? cc : 0);
        a.mup[k] = up;
    }
    a.coff = rowc * U + s;
    const int c = lane < 2 * r ? lane : 0;
    a.bup = c >= r && r > 0;
    const int cc = a.bup ? c - r : c;
    const bool in = r > 0 && row0 + (8 * cc) / r < f;
    a.boff = (r > 0 ? (long)row0 * r / 8 : 0) + (in ? cc : 0);
    return a;
}

template <int KM>
__device__ __forceinline__ void sl_meta_load(uint4 (&meta)[KM], const StackLayer& w, const SlGuAddr<KM>& a) {
#pragma unroll
    for (int k = 0; k < KM; ++k)
        meta[k] = load_stream(reinterpret_cast<const uint4*>(a.mup[k] ? w.mu : w.mg) + a.moff[k]);
}

template <int JG, int KM>
__device__ __forceinline__ void sl_b_load(FGuItem<1, 8, JG, KM>& it, const StackLayer& w, const SlGuAddr<KM>& a,
                                          int r) {
    const uint4* base = r > 0 ? reinterpret_cast<const uint4*>(a.bup ? w.Bu : w.Bg)
                              : reinterpret_cast<const uint4*>(w.cg);
    const uint4 b = load_stream(base + a.boff);
    it.bg[0] = b.x; it.bg[1] = b.y; it.bu[0] = b.z; it.bu[1] = b.w;
}

// sk_gu_accumulate with the next block's codes of slot i requested right
// after slot i's arithmetic (RELOAD), so the gate/up stream of block i+1
// starts while block i's dot products are still running.
template <int JG, int KM, bool RELOAD>
__device__ __forceinline__ void sl_gu_accumulate(FGuItem<1, 8, JG, KM>& it, const uint4* xs, const float2* cx,
                                                 int g, const uint32_t* wmeta, int lane, const StackLayer& wn,
                                                 const SlGuAddr<KM>& a) {
    constexpr int XS = 8 * JG;
    const uint32_t mv = magic_vgpr();
    const int s = lane & 7, r = lane >> 3;
    const int ng = XS * 64 / g, gsh = g == 128 ? 1 : 0;
    const uint4* xl = xs + s;
    const float2* cl = cx + s;
    const uint32_t* mgl = wmeta + r * ng + (s >> gsh);
    const uint32_t* mul = wmeta + (8 + r) * ng + (s >> gsh);
    const uint4* cg = reinterpret_cast<const uint4*>(wn.cg) + a.coff;
    const uint4* cu = reinterpret_cast<const uint4*>(wn.cu) + a.coff;
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
        if constexpr (RELOAD) {
            sk_order();
            it.qg[i] = load_stream(cg + 8 * i);
            it.qu[i] = load_stream(cu + 8 * i);
        }
    }
}

// A gate/up wave: gate/up wave-item `wave` of block i in iteration i; its
// registers are reloaded with block i+1's codes as they fall free (metadata
// once parked in LDS, each slot's codes after its arithmetic, LoRA-B after
// the row sums).  A wave runs one kind of arithmetic only, and its loop body
// issues its loads without a condition (the last block is peeled off), so the
// loads it waits for are always exactly the oldest ones it has in flight.
template <int JG, int KM>
__device__ __forceinline__ void sl_gu_role(const LayersArgs& sa, LKArgs* ka, const SlLds& m, int xcc, int j,
                                           uint32_t seq0, int wave, int lane) {
    const int d = sa.d, f = sa.f, g = sa.g, r = sa.r, L = sa.L;
    const int FX = f / SX, RG = f / SGRID, UG = d / 64;
    const int row_begin = xcc * FX + j * RG, row_end = row_begin + RG;
    const int row0 = row_begin + 8 * wave;
    const SlGuAddr<KM> ga = sl_gu_addr<KM>(row0, row_end, f, d, g, r, lane);
    FGuItem<1, 8, JG, KM> gi;
    sk_gu_load(gi, sk_layer(ka, 0), row0, row_end, f, d, g, r, lane);
    // This wave's h words in all four slots start the launch with tag 0
    // (never a valid tag): a slot that earlier launches left unused for a
    // long time cannot hold a word whose 16-bit tag comes round again.  The
    // same lane publishes the row later, so the clear precedes it.
    if (gi.ok && (lane & 7) == 0) {
#pragma unroll
        for (int s = 0; s < 4; ++s) st_intra32(sa.hb + (long)s * f + gi.row, 0u);
    }
    __syncthreads();                                            // B0: block 0's input staged
    uint4* wmeta = reinterpret_cast<uint4*>(m.meta + wave * sa.meta_bytes);
    auto compute = [&](int i, auto reload) {
        constexpr bool RL = decltype(reload)::value;
        const int par = i & 1;
        const uint32_t step = seq0 + 1 + i;
        const StackLayer wn = sk_layer(ka, RL ? i + 1 : i);
        GateUpArgs gargs{};
        gargs.d = d;
        gargs.g = g;
        fgu_meta_to_lds(gi, gargs, wmeta, lane);
        if constexpr (RL) {
            sk_order();
            sl_meta_load<KM>(gi.meta, wn, ga);
        }
        sl_gu_accumulate<JG, KM, RL>(gi, m.xs + par * 8 * UG, m.cx + par * UG, g,
                                     reinterpret_cast<const uint32_t*>(wmeta), lane, wn, ga);
        sk_gu_finish(gi, m.ts + par * (2 * r + 1), r, sk_layer(ka, i).lora_scale, sa.hb + (long)(step & 3) * f,
                     stag(step), lane, wmeta + 4 * (d / g));
        sk_order();
        if constexpr (RL)
            sl_b_load(gi, wn, ga, r);
    };
    for (int i = 0; i + 1 < L; ++i) {
        compute(i, std::true_type{});
        gi.G[0] = gi.U[0] = 0.0f;
        __syncthreads();                                        // one barrier per iteration
    }
    compute(L - 1, std::false_type{});
    for (int i = L - 1; i < L + 2; ++i) __syncthreads();       // iterations L-1 .. L+1
}

// One down wave-item (8 output rows, 8 lanes per row) with its metadata
// loaded wide: the groups of the XCD's column slice F_x in the item's 8 rows
// are words [cb, cb + 16) of each row's (scale | zero) words, cb = the slice's
// first group rounded down to a multiple of 4; lane l < 32 loads 16-byte chunk
// l & 3 of row l >> 2, and the arithmetic reads each lane's word from LDS.
// (One load per lane for the item, against one 4-byte load per lane and slot.)
template <int JD>
struct SlDn {
    uint4 q[JD];
    uint4 mc;
};

template <int JD>
__device__ __forceinline__ void sl_dn_load(SlDn<JD>& it, const StackLayer& w, int o0, int xcc, int f, int g,
                                           int lane) {
    const int s = lane & 7, FX = f / SX, UF = FX / 32, Uf = f / 32, ngd = f / g;
    const int o = o0 + (lane >> 3);
    const uint4* cd = reinterpret_cast<const uint4*>(w.cd) + (long)o * Uf + xcc * UF;
#pragma unroll
    for (int i = 0; i < JD; ++i) {
        // only the last slot can run past the slice: it re-reads the slice's
        // last unit, and its contribution is dropped
        const int u = i + 1 < JD ? s + 8 * i : (s + 8 * i < UF ? s + 8 * i : UF - 1);
        it.q[i] = load_stream(cd + u);
    }
    const int cb = ((xcc * FX) / g) & ~3;
    const int l32 = lane & 31, w0 = cb + 4 * (l32 & 3);
    const int wc = w0 + 4 <= ngd ? w0 : cb;                      // a chunk past the row re-reads the first
    it.mc = load_stream(reinterpret_cast<const uint4*>(w.md + (long)(o0 + (l32 >> 2)) * ngd + wc));
}

template <int JD>
__device__ __forceinline__ float sl_dn_compute(const SlDn<JD>& it, const uint4* hs, const float2* hcx, int xcc,
                                               int f, int g, int lane, uint4* wm) {
    constexpr int HS = 8 * JD;
    const int FX = f / SX, UF = FX / 32;
    const uint32_t mv = magic_vgpr();
    const int s = lane & 7;
    const int cb = ((xcc * FX) / g) & ~3;
    if (lane < 32)
        wm[lane] = it.mc;
    const uint32_t* wrow = reinterpret_cast<const uint32_t*>(wm) + (lane >> 3) * 16 - cb;
    const uint4* hl = hs + s;
    const float2* cl = hcx + s;
    float Y = 0.0f;
#pragma unroll
    for (int i = 0; i < JD; ++i) {
        const int u = s + 8 * i;
        const int uc = i + 1 < JD ? u : (u < UF ? u : UF - 1);
        uint32_t wv[4] = {it.q[i].x, it.q[i].y, it.q[i].z, it.q[i].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) pin(wv[q]);
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
        const uint32_t mti = wrow[(xcc * FX + 32 * uc) / g];
        const float2 k = cl[8 * i];
        const float c = h2f(mti & 0xFFFFu) * (acc - k.x - h2f(mti >> 16) * k.y);
        if (i + 1 < JD || u < UF)
            Y += c;
    }
    return group_sum<8>(Y);
}

// A down wave with N down wave-items: the items of block i - 2 in iteration
// i.  With DB the registers are double-buffered: block l+1's codes are
// requested when block l's arithmetic starts, a full iteration before they
// are used (the loop is unrolled by two so each buffer is a fixed register
// set, and the tail is peeled, so the loop issues its loads without a
// condition).  Without DB each item's registers are reloaded right after the
// arithmetic.
template <int JD, int N, bool DB>
__device__ __forceinline__ void sl_dn_role(const LayersArgs& sa, LKArgs* ka, const SlLds& m, int xcc, int j,
                                           uint32_t seq0, int wave, int lane) {
    const int d = sa.d, f = sa.f, g = sa.g, L = sa.L;
    const int DJ = d / SB;
    constexpr int HS = 8 * JD;
    const int o0 = j * DJ + 8 * ka->dn_lo[wave];                 // first output row of item 0
    const int o = o0 + (lane >> 3);                             // output row of item 0 on this lane
    uint4* wm = m.dmeta + wave * 4 * 32;                        // 32 chunks per item, up to 4 items
    auto load = [&](SlDn<JD> (&dd)[N], int l) {
        const StackLayer w = sk_layer(ka, l);
#pragma unroll
        for (int k = 0; k < N; ++k) sl_dn_load(dd[k], w, o0 + 8 * k, xcc, f, g, lane);
    };
    // All items' arithmetic first, then their stores: a store counts in the
    // same in-order counter as the loads, so a store between two items would
    // make the second item wait for its completion.
    auto items = [&](SlDn<JD> (&dd)[N], int l) {
        float yv[N];
#pragma unroll
        for (int k = 0; k < N; ++k)
            yv[k] = sl_dn_compute<JD>(dd[k], m.hs + (l & 1) * 4 * HS, m.hcx + (l & 1) * HS, xcc, f, g, lane,
                                      wm + 32 * k);
        const unsigned long long tg = (unsigned long long)ltag32(seq0 + 1 + l) << 32;
#pragma unroll
        for (int k = 0; k < N; ++k)
            if ((lane & 7) == 0)
                st_cross64(sa.pb + ((long)l * SX + xcc) * d + o + 8 * k, (unsigned long long)__float_as_uint(yv[k]) | tg);
        sk_order();
    };
    SlDn<JD> da[N];
    load(da, 0);
    __syncthreads();                                            // B0
    __syncthreads();                                            // iteration 0
    __syncthreads();                                            // iteration 1
    if constexpr (DB) {
        SlDn<JD> db[N];
        int l = 0;                                              // block l is in da
        for (; l + 2 < L; l += 2) {                             // iterations l + 2, l + 3
            load(db, l + 1);
            items(da, l);
            __syncthreads();
            load(da, l + 2);
            items(db, l + 1);
            __syncthreads();
        }
        if (l + 2 == L) {
            load(db, l + 1);
            items(da, l);
            __syncthreads();
            items(db, l + 1);
            __syncthreads();
        } else {
            items(da, l);
            __syncthreads();
        }
    } else {
        for (int l = 0; l + 1 < L; ++l) {                       // iteration l + 2
            items(da, l);
            load(da, l + 1);
            __syncthreads();
        }
        items(da, L - 1);                                       // iteration L + 1
        __syncthreads();
    }
}

// A compute wave without work in this plan: the barriers only.
__device__ __forceinline__ void sl_idle_role(int L) {
    for (int i = 0; i < L + 3; ++i) __syncthreads();           // B0 and L + 2 iterations
}

// After the iterations: every thread of the workgroup sums the eight
// cross-XCD partials of two rows of this workgroup's share of y,
// D_j[xcc DJ/8, (xcc+1) DJ/8), for one block, in XCD order; all blocks' sums
// are polled together (the partials have one slot per block).  Until then
// no XCD waits for another.
__device__ __forceinline__ void sl_sum_y(const LayersArgs& sa, int xcc, int j, uint32_t seq0, int tid, int lane) {
    const int d = sa.d, L = sa.L, DJ = d / SB, PR = DJ / 16;
    const int yrow0 = j * DJ + xcc * (DJ / 8);
    bool dead = false;
    for (int t = tid; t < ((L * PR + 63) & ~63); t += LTHREADS) {   // whole waves per round
        const bool live = t < L * PR;
        const int ly = live ? t / PR : 0, pr = live ? t - ly * PR : 0;
        const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(
            sa.pb + (long)ly * SX * d + yrow0, 0, ((SX - 1) * d + DJ / 8) * 8, 0x00020000);
        int off[SX];
#pragma unroll
        for (int xx = 0; xx < SX; ++xx) off[xx] = 16 * pr + xx * d * 8;
        u32x4 v[SX];
        dead |= !sk_poll<SX, 0, POL_CROSS>(prs, off, live ? 0xFFu : 0u, v, ltag32(seq0 + 1 + ly), dead);
        float y0 = 0.0f, y1 = 0.0f;
#pragma unroll
        for (int xx = 0; xx < SX; ++xx) {
            y0 += __uint_as_float(v[xx].x);
            y1 += __uint_as_float(v[xx].z);
        }
        if (live)
            reinterpret_cast<uint32_t*>(sa.y + (long)ly * d + yrow0)[pr] = f2h(y0) | (f2h(y1) << 16);
    }
    dead = __builtin_amdgcn_readfirstlane(__any(dead) ? 1 : 0) != 0;
    if (dead && lane == 0)
        atomicOr(&sa.ctl[L_ERR], 4u);
}

// The polling waves: the LoRA-A products of every block (once), then per
// iteration the next block's input, h of the previous block, and y of the
// block before that.
template <int XS, int HS>
__device__ __forceinline__ void sl_poll_role(const LayersArgs& sa, LKArgs* ka, const SlLds& m, int xcc, int j,
                                             uint32_t seq0, int wave, int lane) {
    const int d = sa.d, f = sa.f, r = sa.r, L = sa.L;
    const int FX = f / SX;
    const int pw = wave - LCW, pt = pw * 64 + lane;
    unsigned* ctl = sa.ctl;
    bool dead = false;                                          // this wave gave up a wait

    // LoRA-A products: dot product idx = (block l, rank k) on polling wave idx % 512
    if (r > 0) {
        const int total = L * 2 * r;
        for (int idx = (xcc * SB + j) * SPW + pw; idx < total; idx += SGRID * SPW) {
            const int l = idx / (2 * r), k = idx - l * 2 * r;
            const StackLayer w = sk_layer(ka, l);
            const uint16_t* arow = k < r ? w.Ag + (long)k * d : w.Au + (long)(k - r) * d;
            const uint16_t* xl = sa.x + (long)l * d;
            float acc = 0.0f;
            for (int c = lane * 8; c < d; c += 512) {
                const uint4 av = *reinterpret_cast<const uint4*>(arow + c);
                const uint4 xv = *reinterpret_cast<const uint4*>(xl + c);
                acc = dot2(av.x, xv.x, acc);
                acc = dot2(av.y, xv.y, acc);
                acc = dot2(av.z, xv.z, acc);
                acc = dot2(av.w, xv.w, acc);
            }
            acc = group_sum<64>(acc);
            if (lane == 0)
                st_cross64(sa.tb + idx, (unsigned long long)__float_as_uint(acc) |
                                            ((unsigned long long)ltag32(seq0 + 1 + l) << 32));
        }
    }

    const __amdgpu_buffer_rsrc_t trs =
        __builtin_amdgcn_make_buffer_rsrc(sa.tb, 0, kLayersMaxLayers * 2 * (r > 0 ? r : 1) * 8, 0x00020000);
    // h words of this XCD's slice: staging word w = pt + SPT kk covers h[8w, 8w + 8)
    int hoff[2 * KHW];
    uint32_t hvalid = 0;
#pragma unroll
    for (int kk = 0; kk < KHW; ++kk) {
#pragma unroll
        for (int q = 0; q < 2; ++q) hoff[2 * kk + q] = 32 * pt + 32 * SPT * kk + 16 * q;
        if (pt + SPT * kk < FX / 8) hvalid |= 0x3u << (2 * kk);
    }
    // Per iteration the first round of every load (the next block's input
    // and LoRA-A products, h of the previous block) goes out together; then
    // each is resolved in turn.
    uint4 xv[KXW][2];
    u32x4 tv[1];
    int toff[1] = {0};
    auto issue_input = [&](int l) {
        const uint16_t* xl = sa.x + (long)l * d;
#pragma unroll
        for (int kk = 0; kk < KXW; ++kk) {
            const int w = pt + SPT * kk;
            const int wc = w < d / 16 ? w : 0;
            xv[kk][0] = *reinterpret_cast<const uint4*>(xl + 16 * wc);
            xv[kk][1] = *reinterpret_cast<const uint4*>(xl + 16 * wc + 8);
        }
        toff[0] = (l * 2 * r + 2 * pt) * 8;              // ranks 2 pt, 2 pt + 1
        if (r > 0)
            sk_poll_issue<1, POL_CROSS>(trs, toff, pt < r && !dead ? 1u : 0u, tv);
    };
    auto finish_input = [&](int l) {
        const int par = l & 1;
        if (r > 0) {
            if (!dead)
                dead = !sk_poll_finish<1, 0, POL_CROSS>(trs, toff, pt < r ? 1u : 0u, tv, ltag32(seq0 + 1 + l));
            if (pt < r) {
                m.ts[par * (2 * r + 1) + 2 * pt] = __uint_as_float(tv[0].x);
                m.ts[par * (2 * r + 1) + 2 * pt + 1] = __uint_as_float(tv[0].z);
            }
        }
        if (pt == 0)
            m.ts[par * (2 * r + 1) + 2 * r] = 1.0f;
#pragma unroll
        for (int kk = 0; kk < KXW; ++kk) {
            const int w = pt + SPT * kk;
            sl_stage_x<XS>(m.xs + par * 8 * XS, m.cx + par * XS, xv[kk], w < d / 16, w);
        }
        dead = __builtin_amdgcn_readfirstlane(__any(dead) ? 1 : 0) != 0;
        if (dead && lane == 0)
            atomicOr(&ctl[L_ERR], 1u);
    };

    issue_input(0);
    finish_input(0);
    __syncthreads();                                            // B0

    for (int i = 0; i < L + 2; ++i) {
        const int lh = i - 1;
        const bool dx = i + 1 < L, dh = lh >= 0 && lh < L;
        const uint32_t hstep = seq0 + 1 + lh;
        const __amdgpu_buffer_rsrc_t hrs = __builtin_amdgcn_make_buffer_rsrc(
            sa.hb + (long)(hstep & 3) * f + (long)xcc * FX, 0, FX * 4, 0x00020000);
        u32x4 hv[2 * KHW];
        // At the default priority the arithmetic waves on this SIMD would hold
        // the issue slots until their items are done and delay every
        // hand-off; the loads of the iteration and the staging of the next
        // input therefore run at a raised priority, the waits at the default.
        __builtin_amdgcn_s_setprio(3);
        if (dx)
            issue_input(i + 1);
        if (dh && !dead)
            sk_poll_issue<2 * KHW, POL_INTRA>(hrs, hoff, hvalid, hv);
        if (dx)
            finish_input(i + 1);
        __builtin_amdgcn_s_setprio(0);
        if (dh) {   // h of block lh from this XCD
            if (!dead)
                dead = !sk_poll_finish<2 * KHW, 2 * KHW, POL_INTRA>(hrs, hoff, hvalid, hv, stag(hstep));
            const int par = lh & 1;
#pragma unroll
            for (int kk = 0; kk < KHW; ++kk) {
                const int w = pt + SPT * kk;
                sk_stage_h<HS>(m.hs + par * 4 * HS, m.hcx + par * HS, hv + 2 * kk, w < FX / 8, w);
            }
            dead = __builtin_amdgcn_readfirstlane(__any(dead) ? 1 : 0) != 0;
            if (dead && lane == 0)
                atomicOr(&ctl[L_ERR], 2u);
        }
        __syncthreads();
    }
}

template <int JG, int KM, int JD, int NDN>
__global__ void __launch_bounds__(LTHREADS) layers_kernel(LayersArgs sa) {
    extern __shared__ uint4 smem[];
    char* lds = reinterpret_cast<char*>(smem);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    unsigned* ctl = sa.ctl;
    int* info = reinterpret_cast<int*>(lds);

    // Placement: the XCD from the hardware, the rank from a per-XCD counter.
    const uint32_t xcc = __builtin_amdgcn_s_getreg(20 | (0 << 6) | (3 << 11));   // HW_REG_XCC_ID[3:0]
    if (tid == 0)
        info[0] = xcc < (uint32_t)SX ? (int)__hip_atomic_fetch_add(&ctl[L_XC + xcc], 1u, __ATOMIC_RELAXED,
                                                                   __HIP_MEMORY_SCOPE_AGENT)
                                     : SB;
    const uint32_t seq0 = __builtin_amdgcn_readfirstlane(
        __hip_atomic_load(&ctl[L_SEQ], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    __syncthreads();
    const int j = __builtin_amdgcn_readfirstlane(info[0]);

    if (j < SB) {
        const SlLds m{reinterpret_cast<uint4*>(lds + sa.o_xs), reinterpret_cast<float2*>(lds + sa.o_cx),
                      reinterpret_cast<float*>(lds + sa.o_t), reinterpret_cast<uint4*>(lds + sa.o_hs),
                      reinterpret_cast<float2*>(lds + sa.o_hcx), lds + sa.o_meta,
                      reinterpret_cast<uint4*>(lds + sa.o_dmeta)};
        LKArgs* ka = (LKArgs*)__builtin_amdgcn_kernarg_segment_ptr();
        if (wave < sa.n_gu)
            sl_gu_role<JG, KM>(sa, ka, m, (int)xcc, j, seq0, wave, lane);
        else if (wave < LCW) {
            const int n = ka->dn_n[wave];
            if (n == 1)
                sl_dn_role<JD, 1, true>(sa, ka, m, (int)xcc, j, seq0, wave, lane);
            else if (n == 2 && NDN >= 2)
                sl_dn_role<JD, (NDN >= 2 ? 2 : 1), true>(sa, ka, m, (int)xcc, j, seq0, wave, lane);
            else if (n == 3 && NDN >= 3)
                sl_dn_role<JD, (NDN >= 3 ? 3 : 1), false>(sa, ka, m, (int)xcc, j, seq0, wave, lane);
            else if (n == 4 && NDN >= 4)
                sl_dn_role<JD, (NDN >= 4 ? 4 : 1), false>(sa, ka, m, (int)xcc, j, seq0, wave, lane);
            else
                sl_idle_role(sa.L);
        }
        else
            sl_poll_role<8 * JG, 8 * JD>(sa, ka, m, (int)xcc, j, seq0, wave, lane);
        sl_sum_y(sa, (int)xcc, j, seq0, tid, lane);
    } else if (tid == 0) {
        atomicOr(&ctl[L_ERR], 8u);              // a workgroup without a place: results invalid
    }

    // The last workgroup to finish advances the step counter and clears the
    // placement counters.
    if (tid == 0) {
        const unsigned old = __hip_atomic_fetch_add(&ctl[L_DONE], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (old == (unsigned)gridDim.x - 1) {
            __hip_atomic_store(&ctl[L_DONE], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (int x = 0; x < SX; ++x)
                __hip_atomic_store(&ctl[L_XC + x], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&ctl[L_SEQ], seq0 + (uint32_t)sa.L + 1u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

int layers_cu_count() {
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

struct LayersPlan {
    int jg, km, jd, ndn;
    int n_gu, dn_lo[LCW], dn_n[LCW];
    int o_xs, o_cx, o_t, o_hs, o_hcx, o_meta, meta_bytes, o_dmeta;
    size_t lds;
    bool ok;
};

// Wave plan: gate/up wave-item k on compute wave k; the down items go one at
// a time to the SIMD with the least dequant work (waves w and w + 4 share a
// SIMD; a gate/up item weighs 12 d / f down items -- 8 rows of 2 d two-bit
// weights against 8 rows of f/8 four-bit weights, scaled so that at
// d = 2560, f = 9728 the SIMD of two gate/up waves gets no down item, which
// measured fastest; a polling wave weighs one), on its down wave
// with the fewest items below the register limit; each wave's items are then
// numbered consecutively.
void plan_waves(LayersPlan& p, int gu_items, int dn_items, int d, int f) {
    const double rho = 12.0 * d / f;
    double load[4] = {0.0, 0.0, 0.0, 0.0};
    load[LCW & 3] += 1.0;                                       // the polling waves
    load[(LCW + 1) & 3] += 1.0;
    int cnt[LCW] = {};
    p.n_gu = gu_items;
    for (int w = 0; w < gu_items; ++w) load[w & 3] += rho;
    for (int it = 0; it < dn_items; ++it) {
        int best = -1;
        for (int w = gu_items; w < LCW; ++w) {
            if (cnt[w] >= p.ndn)
                continue;
            if (best < 0 || load[w & 3] < load[best & 3] ||
                (load[w & 3] == load[best & 3] && cnt[w] < cnt[best]))
                best = w;
        }
        if (best < 0) {
            p.ok = false;
            return;
        }
        ++cnt[best];
        load[best & 3] += 1.0;
    }
    int lo = 0;
    for (int w = 0; w < LCW; ++w) {
        p.dn_lo[w] = lo;
        p.dn_n[w] = cnt[w];
        lo += cnt[w];
    }
}

LayersPlan plan_layers(int M, int d, int f, int g, int r) {
    LayersPlan p{};
    p.ok = false;
    if (M != 1 || d <= 0 || f <= 0 || (g != 64 && g != 128))
        return p;
    if (f % SGRID != 0 || (f / SX) % 32 != 0 || d % 512 != 0 || d % g != 0 || f % g != 0)
        return p;
    const int RG = f / SGRID, UG = d / 64, ng = d / g, UF = f / SX / 32, DJ = d / SB;
    if ((RG + 7) / 8 > LGU_MAX || ng % 4 != 0 || DJ % 16 != 0 || DJ / 16 > 64)
        return p;
    // down metadata: rows 16-byte aligned, and each XCD slice's groups inside a
    // 16-word window that starts at a multiple of 4
    if ((f / g) % 4 != 0)
        return p;
    for (int x = 0; x < SX; ++x) {
        const int lo = x * (f / SX) / g, hi = ((x + 1) * (f / SX) - 1) / g;
        if (hi - (lo & ~3) >= 16)
            return p;
    }
    if (r != 0 && r != 8 && r != 16 && r != 32)
        return p;
    if (UG % 8 != 0)                             // 8 lanes per row, no partial slot
        return p;
    p.jg = UG / 8;
    p.km = (4 * ng + 63) / 64;
    p.jd = (UF + 7) / 8;
    if ((d / 16 + SPT - 1) / SPT > KXW || (f / SX / 8 + SPT - 1) / SPT > KHW)
        return p;
    if (p.jg == 5 && p.km == 2 && p.jd == 5)
        p.ndn = 3;
    else if (p.jg == 8 && p.km == 2 && p.jd == 6)
        p.ndn = 4;
    else if (p.jg == 1 && p.km == 1 && p.jd == 1)
        p.ndn = 1;
    else
        return p;
    if (layers_cu_count() != SGRID)
        return p;
    p.ok = true;
    plan_waves(p, (RG + 7) / 8, DJ / 8, d, f);
    if (!p.ok)
        return p;
    size_t o = 16;
    auto take = [&](size_t bytes) { const size_t at = o; o = (o + bytes + 15) / 16 * 16; return (int)at; };
    p.o_xs = take((size_t)2 * UG * 8 * 16);
    p.o_cx = take((size_t)2 * UG * 8);
    p.o_t = take((size_t)2 * (2 * r + 1) * 4);
    p.o_hs = take((size_t)2 * p.jd * 8 * 4 * 16);   // chunk stride 8 JD >= UF units
    p.o_hcx = take((size_t)2 * p.jd * 8 * 8);
    p.meta_bytes = 2 * 8 * ng * 4 + 32 * r;      // metadata, then LoRA-B rows
    p.o_meta = take((size_t)LGU_MAX * p.meta_bytes);
    p.o_dmeta = take((size_t)LCW * 4 * 32 * 16);
    p.lds = o;
    p.ok = p.lds <= 64 * 1024;
    return p;
}

size_t tb_bytes(int r) { return ((size_t)kLayersMaxLayers * 2 * (r > 0 ? r : 1) * 8 + 255) & ~(size_t)255; }

}  // namespace

bool layers_supported(int M, int d, int f, int g, int r) { return plan_layers(M, d, f, g, r).ok; }

size_t layers_ws_bytes(int d, int f, int r) {
    return 1024 + tb_bytes(r) + (((size_t)4 * f * 4 + 255) & ~(size_t)255) +
           (size_t)kLayersMaxLayers * SX * d * 8;
}

int layers_max_layers() { return kLayersMaxLayers; }

hipError_t launch_layers(const StackLayerDesc* layers, int L, int d, int f, int g, int r, const uint16_t* x,
                         uint16_t* y, void* ws, hipStream_t st) {
    const LayersPlan p = plan_layers(1, d, f, g, r);
    if (!p.ok || L <= 0 || L > kLayersMaxLayers)
        return hipErrorInvalidValue;
    LayersArgs a{};
    for (int i = 0; i < L; ++i) {
        const StackLayerDesc& s = layers[i];
        a.lay[i] = StackLayer{s.cg, s.mg, s.cu, s.mu, s.cd, s.md, s.Bg, s.Bu, s.Ag, s.Au, s.lora_scale};
    }
    a.L = L;
    a.d = d;
    a.f = f;
    a.g = g;
    a.r = r;
    a.x = x;
    a.y = y;
    char* base = static_cast<char*>(ws);
    a.ctl = reinterpret_cast<unsigned*>(base);
    a.tb = reinterpret_cast<unsigned long long*>(base + 1024);
    a.hb = reinterpret_cast<uint32_t*>(base + 1024 + tb_bytes(r));
    a.pb = reinterpret_cast<unsigned long long*>(base + 1024 + tb_bytes(r) +
                                                 (((size_t)4 * f * 4 + 255) & ~(size_t)255));
    a.n_gu = p.n_gu;
    for (int w = 0; w < LCW; ++w) {
        a.dn_lo[w] = p.dn_lo[w];
        a.dn_n[w] = p.dn_n[w];
    }
    a.o_xs = p.o_xs; a.o_cx = p.o_cx; a.o_t = p.o_t; a.o_hs = p.o_hs; a.o_hcx = p.o_hcx;
    a.o_meta = p.o_meta; a.meta_bytes = p.meta_bytes; a.o_dmeta = p.o_dmeta;
    auto run = [&](auto kernel) -> hipError_t {
        kernel<<<SGRID, LTHREADS, p.lds, st>>>(a);
        return hipGetLastError();
    };
    if (p.jg == 5)
        return run(layers_kernel<5, 2, 5, 3>);
    if (p.jg == 8)
        return run(layers_kernel<8, 2, 6, 4>);
    return run(layers_kernel<1, 1, 1, 1>);
}

}  // namespace qmlp

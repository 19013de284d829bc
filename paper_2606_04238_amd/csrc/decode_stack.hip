// A stack of decode MLP blocks in one persistent launch (M = 1, binary16),
// gfx950.
//
// Each block of the stack is the W4/W2-GateUp MLP with Recover-LoRA
// adapters (Sec. 3.1 Eq. (1), Sec. 3.3, Sec. 4.2):
//   G = W2gate x + s B_g (A_g x),  U = W2up x + s B_u (A_u x),
//   h = SiLU(G) * U,  y = W4down h,
// and the blocks sit on a residual stream as in a decoder: block l reads
// u_l = RMSNorm(x_l) (unit gain: a learned gain folds into the block's
// input columns before quantization) and x_{l+1} = x_l + y_l (each y_l
// rounded to binary16 and returned, the sum rounded once), with the
// attention blocks left out.  Decode is bound by loading
// weights (Sec. 3.3, Sec. 5); what a per-layer launch cannot hide is the
// chain of dependent steps inside a layer.  Here the weights of block l+1
// stream into registers while block l runs its hand-offs: weights do not
// depend on activations, so every register set is reloaded with the next
// block's weights right after its last use.  No step of block l+1 starts
// before block l's output is complete.
//
// Work split (8 XCDs x 32 compute units, one 512-thread workgroup each):
//   * XCD x owns the slice F_x = [x f/8, (x+1) f/8) of the intermediate
//     dimension.  Its block j computes gate/up rows F_x,j (f/256 rows) and
//     publishes h for them to the other blocks of the same XCD;
//   * block j then computes the partial down product over F_x for the
//     output rows D_j = [j d/32, (j+1) d/32) and publishes it to the blocks
//     j of the other XCDs;
//   * block j of every XCD sums the eight partials of D_j in XCD order (the
//     same sum on every XCD), rounds y to binary16, adds the residual
//     x[D_j], computes its shares of the next block's LoRA-A product
//     (A[:, D_j] x_{l+1}[D_j], fp32) and of sum x_{l+1}^2 over D_j, and
//     publishes them with x_{l+1}[D_j] to the blocks of its own XCD, which
//     add the 32 shares in order; the norm then scales the staged input, and
//     the LoRA-A product by the same factor (it is linear in the input).
// So every layer has one hand-off between XCDs and two inside an XCD,
// through that XCD's L2.  The XCD of a workgroup is read from HW_REG_XCC_ID
// and its rank inside the XCD from a per-XCD counter, so producer and
// consumer of an XCD-local word are on the same L2 by construction.
//
// Hand-offs carry their own validity: each published value sits in one
// aligned word with a tag that changes with every layer step (32-bit words:
// binary16 | 16-bit tag << 16; 64-bit words: fp32 bits | tag << 32, the
// cross-XCD partials with a 32-bit tag, since a slot of their parity-double
// buffer can go unwritten for many launches of one layer).  XCD-local words
// are written with plain stores and polled with sc0|nt loads (they miss the
// CU's L1 and hit the XCD's L2); cross-XCD words are written and polled
// device-coherent (sc1), double-buffered by layer parity (an XCD can run at
// most one layer ahead of another).  Waves 0-5 hold and
// stream weights and compute; waves 6-7 only poll, so their polls are never
// queued behind the weight stream of their own wave.  Every wait is bounded:
// a timeout sets an error bit, later polls of that wave are skipped and the
// kernel exits normally.
#include "stack_common.h"

namespace qmlp {

namespace {

constexpr int KA = 3;                     // LoRA-A slice loads per compute thread (max)
constexpr float kRmsEps = 1e-6f;          // RMSNorm epsilon
// Where the next layer's gate/up codes are requested: 0 right after this
// layer's gate/up arithmetic, 1 after the down arithmetic (with the down
// codes), 2 after the last barrier of the layer.  A burst of requests delays
// the hand-off polls issued behind it on the same compute unit, so the
// choice decides which hand-off overlaps the gate/up half of the stream.
constexpr int kGuPrefetchAt = 0;

}  // namespace

constexpr int kStackMaxLayers = 40;            // layers per launch (kernel-argument block < 4 KB)

struct StackArgs {
    StackLayer lay[kStackMaxLayers];
    int L, d, f, g, r;
    const uint16_t* x0;          // [d] input of the first layer
    uint16_t* y;                 // [L][d] output of every layer
    uint16_t* xl;                // [d] the residual stream after the last layer (may be null)
    uint32_t* xb;                // [8][xw] XCD-local, 64-bit tagged words: x' pairs [d/2], per-word
                                 // sums [d/8], shares [2r+1][32] (LoRA-A ranks, sum of squares)
    uint32_t* hb;                // [f] XCD-local h words (XCD x owns [x f/8, (x+1) f/8))
    unsigned long long* pb;      // [2][8][d] cross-XCD partial down sums
    unsigned* ctl;
    int xw;                      // 32-bit words per XCD in xb
    int o_xs, o_cx, o_t, o_hs, o_hcx, o_a, o_y, o_xn, o_meta, meta_bytes;   // LDS byte offsets
};

namespace {

// The LoRA-A columns D_j of the next layer, [2r][DJ] binary16 (gate ranks
// then up ranks), KA 16-byte pieces per compute thread.
__device__ __forceinline__ void sk_a_load(uint4 (&av)[KA], const StackLayer& w, int r, int d, int DJ,
                                          int j, int ct) {
    const int per = DJ / 8, total = 2 * r * per;
#pragma unroll
    for (int k = 0; k < KA; ++k) {
        const int q = ct + SCW * 64 * k;
        const int qq = q < total ? q : 0;
        const int rk = qq / per, c8 = qq - rk * per;
        const uint16_t* row = rk < r ? w.Ag + (long)rk * d : w.Au + (long)(rk - r) * d;
        if (total > 0)
            av[k] = *reinterpret_cast<const uint4*>(row + j * DJ + 8 * c8);
    }
}

__device__ __forceinline__ void sk_a_store(const uint4 (&av)[KA], uint4* as, int r, int DJ, int ct) {
    const int total = 2 * r * (DJ / 8);
#pragma unroll
    for (int k = 0; k < KA; ++k) {
        const int q = ct + SCW * 64 * k;
        if (q < total)
            as[q] = av[k];
    }
}

// Polling wave 0: block j's rows D_j of the next layer's stream x (binary16
// pairs (2l, 2l+1) in xn, LDS) go to the XCD-local activation buffer already
// in the gate/up x' layout, so consumers only move words into LDS:
//   * staging word w (16 values) holds pairs p = 0..7 of (x[16w+p],
//     x[16w+8+p]), each half pre-scaled by its fraction position, as
//     64-bit words pair | tag << 32 at [8w + p];
//   * its sums (1024 sum x', sum x) as two tagged 64-bit words at
//     [d/2 + 2w], [d/2 + 2w + 1];
//   * block j's shares of A x (per rank, unnormalized) and of sum x^2 at
//     [d/2 + d/8 + k 32 + j] (k = 2r: the sum of squares).
// Lane l < DJ/2 covers staging word l / 8 of D_j, pair l % 8.
__device__ __forceinline__ void sk_publish_x(uint32_t* xb, const uint32_t* xn, const uint16_t* as,
                                             int d, int r, int DJ, int j, uint32_t tag, int lane) {
    unsigned long long* x64 = reinterpret_cast<unsigned long long*>(xb);
    const unsigned long long tg = (unsigned long long)tag << 32;
    const uint16_t* xh = reinterpret_cast<const uint16_t*>(xn);
    const bool live = lane < DJ / 2;
    const int wl = lane >> 3, p = lane & 7;
    const uint32_t a = live ? xh[16 * wl + p] : 0u, b = live ? xh[16 * wl + 8 + p] : 0u;
    const float sc = w2_pair_scale(p);
    const uint32_t ha = f2h(h2f(a) * sc), hb = f2h(h2f(b) * sc);
    const int gw = j * (DJ / 16) + wl;
    if (live)
        st_intra64(x64 + 8 * gw + p, (unsigned long long)(ha | (hb << 16)) | tg);
    const float cs = group_sum<8>(h2f(ha) + h2f(hb));
    const float xs = group_sum<8>(h2f(a) + h2f(b));
    if (live && p == 0) {
        st_intra64(x64 + d / 2 + 2 * gw, (unsigned long long)__float_as_uint(1024.0f * cs) | tg);
        st_intra64(x64 + d / 2 + 2 * gw + 1, (unsigned long long)__float_as_uint(xs) | tg);
    }
    unsigned long long* sh = x64 + d / 2 + d / 8;
    // shares of A x: lanes in groups of 64 / 2r per rank, each over a
    // contiguous run of pairs read 16 bytes at a time
    if (r > 0) {
        const int lpr = 64 / (2 * r), k = lane / lpr, sub = lane - k * lpr;
        const int ppl = DJ / 2 / lpr;                          // pairs per lane
        const uint32_t* a32 = reinterpret_cast<const uint32_t*>(as) + k * (DJ / 2) + sub * ppl;
        const uint32_t* x32 = xn + sub * ppl;
        float acc = 0.0f;
        if ((ppl & 3) == 0) {
#pragma unroll 4
            for (int c = 0; c < ppl; c += 4) {
                const uint4 av = *reinterpret_cast<const uint4*>(a32 + c);
                const uint4 xv = *reinterpret_cast<const uint4*>(x32 + c);
                acc = dot2(av.x, xv.x, acc);
                acc = dot2(av.y, xv.y, acc);
                acc = dot2(av.z, xv.z, acc);
                acc = dot2(av.w, xv.w, acc);
            }
        } else {
            for (int c = 0; c < ppl; ++c)
                acc = dot2(a32[c], x32[c], acc);
        }
        if (lpr >= 2) acc += dpp<DPP_QUAD_XOR1>(acc);
        if (lpr >= 4) acc += dpp<DPP_QUAD_XOR2>(acc);
        if (sub == 0)
            st_intra64(sh + k * SB + j, (unsigned long long)__float_as_uint(acc) | tg);
    }
    // the share of sum x^2 (for the next block's norm)
    float ss = 0.0f;
    if (live) {
        const uint32_t v = xn[lane];
        const float u0 = h2f(v & 0xFFFFu), u1 = h2f(v >> 16);
        ss = u0 * u0 + u1 * u1;
    }
    ss = group_sum<64>(ss);
    if (lane == 0)
        st_intra64(sh + 2 * r * SB + j, (unsigned long long)__float_as_uint(ss) | tg);
}


typedef const StackArgs __attribute__((address_space(4))) KArgs;

struct SkLds {
    uint4* xs;          // x' of the activation (gate/up units)
    float2* cxg;        // per unit (1024 sum x', sum x)
    float* ts;          // [A_g; A_u] x (unnormalized), fp32 [2r], then 1 / rms
    uint4* hs;          // h' of this XCD's slice (down units)
    float2* hcx;        // per unit (1024 sum h', sum h)
    uint4* as;          // next layer's LoRA-A columns D_j, binary16 [2r][DJ]
    uint32_t* ys;       // y[D_j] binary16 pairs
    uint32_t* xn;       // the stream x[D_j], binary16 pairs (current, then next layer)
    char* meta;         // per-wave gate/up metadata areas
};

struct SkPlace {
    int xcc, j;
    uint32_t seq0;
};

// The weight waves: stream every layer's weights into registers (each set
// reloaded for the next layer right after its last use), compute gate/up
// rows and the partial down sums.  One barrier before the layers and three
// per layer, matching sk_poll_role.
template <int JG, int KM, int JD, int NDN>
__device__ __forceinline__ void sk_compute_role(const StackArgs& sa, KArgs* ka, const SkLds& m,
                                                const SkPlace& pl, int wave, int lane) {
    const int d = sa.d, f = sa.f, g = sa.g, r = sa.r, L = sa.L;
    const int FX = f / SX, UF = FX / 32, DJ = d / SB, RG = f / SGRID;
    const int xcc = pl.xcc, j = pl.j, ct = wave * 64 + lane;
    const int row_begin = xcc * FX + j * RG, row_end = row_begin + RG;
    const int gu_items = (RG + 7) / 8, dn_items = DJ / 8;
    const bool has_gu = wave < gu_items;
    FGuItem<1, 8, JG, KM> gi;
    SkDn<JD> di[NDN];
    uint4 av[KA];
    {
        const StackLayer w0 = sk_layer(ka, 0);
        sk_a_load(av, w0, r, d, DJ, j, ct);
        if (has_gu)
            sk_gu_load(gi, w0, row_begin + 8 * wave, row_end, f, d, g, r, lane);
#pragma unroll
        for (int k = 0; k < NDN; ++k) {
            const int item = wave + SCW * k;
            if (item < dn_items)
                sk_dn_load(di[k], w0, j * DJ + 8 * item + (lane >> 3), xcc, f, g, lane);
        }
        sk_a_store(av, m.as, r, DJ, ct);
    }
    __syncthreads();                                            // B0
    uint4* wmeta = reinterpret_cast<uint4*>(m.meta + wave * sa.meta_bytes);
    for (int i = 0; i < L; ++i) {
        const uint32_t ti = stag(pl.seq0 + 1 + i);
        __syncthreads();                                        // B1: x', t staged
        if (has_gu) {
            GateUpArgs ga{};
            ga.d = d;
            ga.g = g;
            fgu_meta_to_lds(gi, ga, wmeta, lane);
            sk_gu_accumulate(gi, m.xs, m.cxg, g, reinterpret_cast<const uint32_t*>(wmeta), lane);
            sk_gu_finish(gi, m.ts, r, sk_layer(ka, i).lora_scale, sa.hb, ti, lane, wmeta + 4 * (d / g));
        }
        sk_order();
        if (i + 1 < L) {
            const StackLayer wn = sk_layer(ka, i + 1);
            sk_a_load(av, wn, r, d, DJ, j, ct);
            if (has_gu && kGuPrefetchAt == 0)
                sk_gu_load(gi, wn, row_begin + 8 * wave, row_end, f, d, g, r, lane);
        }
        __syncthreads();                                        // B2: h' staged
        unsigned long long* pb = sa.pb + (long)(i & 1) * SX * d + (long)xcc * d;
#pragma unroll
        for (int k = 0; k < NDN; ++k) {
            const int item = wave + SCW * k;
            if (item < dn_items) {
                const float yv = sk_dn_compute<JD>(di[k], m.hs, m.hcx, UF, lane);
                const int o = j * DJ + 8 * item + (lane >> 3);
                if ((lane & 7) == 0)
                    st_cross64(pb + o, (unsigned long long)__float_as_uint(yv) | ((unsigned long long)ltag32(pl.seq0 + 1 + i) << 32));
            }
        }
        sk_order();
        if (i + 1 < L) {
            const StackLayer wn = sk_layer(ka, i + 1);
            sk_a_store(av, m.as, r, DJ, ct);
#pragma unroll
            for (int k = 0; k < NDN; ++k) {
                const int item = wave + SCW * k;
                if (item < dn_items)
                    sk_dn_load(di[k], wn, j * DJ + 8 * item + (lane >> 3), xcc, f, g, lane);
            }
            if (has_gu && kGuPrefetchAt == 1)
                sk_gu_load(gi, wn, row_begin + 8 * wave, row_end, f, d, g, r, lane);
        }
        __syncthreads();                                        // B3: y[D_j], next A in LDS
        if (i + 1 < L && has_gu && kGuPrefetchAt == 2)
            sk_gu_load(gi, sk_layer(ka, i + 1), row_begin + 8 * wave, row_end, f, d, g, r, lane);
    }
}

// The polling waves: move the activation (published in the x' layout) and
// the shares into LDS, stage h, then sum the cross-XCD partials, add the
// residual and publish the next layer's stream rows and shares.
// Offsets of the polled words are affine in the lane (one base register);
// which of them exist is a bit mask.
template <int XS, int HS>
__device__ __forceinline__ void sk_poll_role(const StackArgs& sa, const SkLds& m, const SkPlace& pl,
                                             int wave, int lane) {
    const int d = sa.d, f = sa.f, r = sa.r, L = sa.L;
    const int FX = f / SX, DJ = d / SB;
    const int xcc = pl.xcc, j = pl.j, pt = (wave - SCW) * 64 + lane;
    unsigned* ctl = sa.ctl;
    uint32_t* xb = sa.xb + (long)xcc * sa.xw;
    const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(xb, 0, sa.xw * 4, 0x00020000);
    const __amdgpu_buffer_rsrc_t hrs =
        __builtin_amdgcn_make_buffer_rsrc(sa.hb + (long)xcc * FX, 0, FX * 4, 0x00020000);
    bool dead = false;                                          // this wave gave up a wait
    if (wave == SCW && lane < DJ / 2)
        m.xn[lane] = reinterpret_cast<const uint32_t*>(sa.x0 + j * DJ)[lane];
    __syncthreads();                                            // B0
    if (wave == SCW)
        sk_publish_x(xb, m.xn, reinterpret_cast<const uint16_t*>(m.as), d, r, DJ, j, stag(pl.seq0), lane);

    // activation: staging word w = pt + SPT kk in the x' layout (four 16-byte
    // words of tagged pairs and one of tagged sums); shares of rank pt <= 2r
    // (2r: the sum of squares), 32 64-bit words
    int xoff[5 * KXW + 16];
    uint32_t xvalid = 0;
#pragma unroll
    for (int kk = 0; kk < KXW; ++kk) {
#pragma unroll
        for (int q = 0; q < 4; ++q) xoff[5 * kk + q] = 64 * (pt + SPT * kk) + 16 * q;
        xoff[5 * kk + 4] = 4 * d + 16 * (pt + SPT * kk);
        if (pt + SPT * kk < d / 16) xvalid |= 0x1Fu << (5 * kk);
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) xoff[5 * KXW + q] = (d / 2 + d / 8 + pt * SB) * 8 + 16 * q;
    if (pt <= 2 * r) xvalid |= 0xFFFFu << (5 * KXW);
    // h words of this XCD's slice: staging word w = pt + SPT kk covers h[8w, 8w+8)
    int hoff[2 * KHW];
    uint32_t hvalid = 0;
#pragma unroll
    for (int kk = 0; kk < KHW; ++kk) {
#pragma unroll
        for (int q = 0; q < 2; ++q) hoff[2 * kk + q] = 32 * pt + 32 * SPT * kk + 16 * q;
        if (pt + SPT * kk < FX / 8) hvalid |= 0x3u << (2 * kk);
    }

    for (int i = 0; i < L; ++i) {
        const uint32_t tx = stag(pl.seq0 + i), ti = stag(pl.seq0 + 1 + i);
        {   // the activation (already in the x' layout) and the shares of this XCD
            u32x4 v[5 * KXW + 16];
            dead |= !sk_poll<5 * KXW + 16, 0, POL_INTRA>(xrs, xoff, xvalid, v, tx, dead);
#pragma unroll
            for (int kk = 0; kk < KXW; ++kk) {
                const int w = pt + SPT * kk;
                const bool valid = w < d / 16;
                const u32x4* vw = v + 5 * kk;
                const float cs = group_sum<4>(valid ? __uint_as_float(vw[4].x) : 0.0f);
                const float xs = group_sum<4>(valid ? __uint_as_float(vw[4].z) : 0.0f);
                if (valid) {
                    const int ul = w >> 2, wi = w & 3;
                    m.xs[(2 * wi) * XS + ul] = make_uint4(vw[0].x, vw[0].z, vw[1].x, vw[1].z);
                    m.xs[(2 * wi + 1) * XS + ul] = make_uint4(vw[2].x, vw[2].z, vw[3].x, vw[3].z);
                    if (wi == 0)
                        m.cxg[ul] = make_float2(cs, xs);
                }
            }
            if (pt <= 2 * r) {   // shares in block order; thread 2r: 1 / rms
                float share = 0.0f;
#pragma unroll
                for (int q = 0; q < 16; ++q) {
                    share += __uint_as_float(v[5 * KXW + q].x);
                    share += __uint_as_float(v[5 * KXW + q].z);
                }
                m.ts[pt] = pt < 2 * r ? share : 1.0f / __fsqrt_rn(share / (float)d + kRmsEps);
            }
            dead = __builtin_amdgcn_readfirstlane(__any(dead) ? 1 : 0) != 0;
            if (dead && lane == 0)
                atomicOr(&ctl[C_ERR], 1u);
        }
        __syncthreads();                                        // B1
        {   // h of this XCD's slice
            u32x4 v[2 * KHW];
            dead |= !sk_poll<2 * KHW, 2 * KHW, POL_INTRA>(hrs, hoff, hvalid, v, ti, dead);
#pragma unroll
            for (int kk = 0; kk < KHW; ++kk) {
                const int w = pt + SPT * kk;
                sk_stage_h<HS>(m.hs, m.hcx, v + 2 * kk, w < FX / 8, w);
            }
            dead = __builtin_amdgcn_readfirstlane(__any(dead) ? 1 : 0) != 0;
            if (dead && lane == 0)
                atomicOr(&ctl[C_ERR], 2u);
        }
        __syncthreads();                                        // B2
        if (wave == SCW) {   // the eight partials of rows D_j, summed in XCD order
            const __amdgpu_buffer_rsrc_t prs = __builtin_amdgcn_make_buffer_rsrc(
                sa.pb + (long)(i & 1) * SX * d + j * DJ, 0, (SX - 1) * d * 8 + DJ * 8, 0x00020000);
            int off[SX];
#pragma unroll
            for (int xx = 0; xx < SX; ++xx) off[xx] = 16 * lane + xx * d * 8;
            u32x4 v[SX];
            dead |= !sk_poll<SX, 0, POL_CROSS>(prs, off, lane < DJ / 2 ? 0xFFu : 0u, v, ltag32(pl.seq0 + 1 + i), dead);
            float y0 = 0.0f, y1 = 0.0f;
#pragma unroll
            for (int xx = 0; xx < SX; ++xx) {
                y0 += __uint_as_float(v[xx].x);
                y1 += __uint_as_float(v[xx].z);
            }
            if (lane < DJ / 2)
                m.ys[lane] = f2h(y0) | (f2h(y1) << 16);
            dead = __builtin_amdgcn_readfirstlane(__any(dead) ? 1 : 0) != 0;
            if (dead && lane == 0)
                atomicOr(&ctl[C_ERR], 4u);
        }
        __syncthreads();                                        // B3
        if (wave == SCW) {
            if (lane < DJ / 2) {
                // x_{l+1} = x_l + y_l: two binary16 values summed exactly in fp32, rounded once
                const uint32_t yv = m.ys[lane], xv = m.xn[lane];
                const uint32_t nv = f2h(h2f(xv & 0xFFFFu) + h2f(yv & 0xFFFFu)) |
                                    (f2h(h2f(xv >> 16) + h2f(yv >> 16)) << 16);
                m.xn[lane] = nv;
                if (xcc == 0) {
                    reinterpret_cast<uint32_t*>(sa.y + (long)i * d + j * DJ)[lane] = yv;
                    if (i + 1 == L && sa.xl)
                        reinterpret_cast<uint32_t*>(sa.xl + j * DJ)[lane] = nv;
                }
            }
            if (i + 1 < L)
                sk_publish_x(xb, m.xn, reinterpret_cast<const uint16_t*>(m.as), d, r, DJ, j, ti, lane);
        }
    }
}

template <int JG, int KM, int JD, int NDN>
__global__ void __launch_bounds__(STHREADS) stack_kernel(StackArgs sa) {
    extern __shared__ uint4 smem[];
    char* lds = reinterpret_cast<char*>(smem);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    unsigned* ctl = sa.ctl;
    int* info = reinterpret_cast<int*>(lds);

    // Placement: the XCD from the hardware, the rank from a per-XCD counter.
    const uint32_t xcc = __builtin_amdgcn_s_getreg(20 | (0 << 6) | (3 << 11));   // HW_REG_XCC_ID[3:0]
    if (tid == 0)
        info[0] = xcc < (uint32_t)SX ? (int)__hip_atomic_fetch_add(&ctl[C_XC + xcc], 1u, __ATOMIC_RELAXED,
                                                                   __HIP_MEMORY_SCOPE_AGENT)
                                     : SB;
    const uint32_t seq0 = __builtin_amdgcn_readfirstlane(
        __hip_atomic_load(&ctl[C_SEQ], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    __syncthreads();
    const int j = __builtin_amdgcn_readfirstlane(info[0]);

    if (j < SB) {
        const SkLds m{reinterpret_cast<uint4*>(lds + sa.o_xs), reinterpret_cast<float2*>(lds + sa.o_cx),
                      reinterpret_cast<float*>(lds + sa.o_t), reinterpret_cast<uint4*>(lds + sa.o_hs),
                      reinterpret_cast<float2*>(lds + sa.o_hcx), reinterpret_cast<uint4*>(lds + sa.o_a),
                      reinterpret_cast<uint32_t*>(lds + sa.o_y), reinterpret_cast<uint32_t*>(lds + sa.o_xn),
                      lds + sa.o_meta};
        const SkPlace pl{(int)xcc, j, seq0};
        if (wave < SCW)
            sk_compute_role<JG, KM, JD, NDN>(sa, (KArgs*)__builtin_amdgcn_kernarg_segment_ptr(), m, pl, wave, lane);
        else
            sk_poll_role<8 * JG, 8 * JD>(sa, m, pl, wave, lane);
    } else if (tid == 0) {
        atomicOr(&ctl[C_ERR], 8u);              // a workgroup without a place: results invalid
    }

    // The last workgroup to finish advances the step counter and clears the
    // placement counters.
    if (tid == 0) {
        const unsigned old = __hip_atomic_fetch_add(&ctl[C_DONE], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (old == (unsigned)gridDim.x - 1) {
            __hip_atomic_store(&ctl[C_DONE], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            for (int x = 0; x < SX; ++x)
                __hip_atomic_store(&ctl[C_XC + x], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&ctl[C_SEQ], seq0 + (uint32_t)sa.L + 1u, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// out = x + y elementwise, the exact fp32 sum of two binary16 (bfloat16)
// values rounded once to nearest-even: the residual stream between blocks on
// the per-layer path.
__global__ void residual_kernel(const uint16_t* x, const uint16_t* y, uint16_t* out, int n, int bf16) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n)
        return;
    if (bf16) {
        const float v = __uint_as_float((uint32_t)x[i] << 16) + __uint_as_float((uint32_t)y[i] << 16);
        const uint32_t u = __float_as_uint(v);
        out[i] = (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
    } else {
        out[i] = (uint16_t)f2h(h2f(x[i]) + h2f(y[i]));
    }
}

// u = x / sqrt(mean(x^2) + eps) per row (binary16 in and out; fp32 sums in
// a fixed order): the input of a block on the per-layer path.
__global__ void __launch_bounds__(256) rmsnorm_kernel(const uint16_t* x, uint16_t* u, int d) {
    __shared__ float part[256];
    const uint16_t* xr = x + (long)blockIdx.x * d;
    float ss = 0.0f;
    for (int i = threadIdx.x; i < d; i += 256) {
        const float v = h2f(xr[i]);
        ss += v * v;
    }
    part[threadIdx.x] = ss;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s)
            part[threadIdx.x] += part[threadIdx.x + s];
        __syncthreads();
    }
    const float inv = 1.0f / __fsqrt_rn(part[0] / (float)d + kRmsEps);
    for (int i = threadIdx.x; i < d; i += 256)
        u[(long)blockIdx.x * d + i] = (uint16_t)f2h(h2f(xr[i]) * inv);
}

int stack_cu_count() {
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

struct StackPlan {
    int jg, km, jd, ndn;
    int o_xs, o_cx, o_t, o_hs, o_hcx, o_a, o_y, o_xn, o_meta, meta_bytes;
    size_t lds;
    bool ok;
};

StackPlan plan_stack(int M, int d, int f, int g, int r) {
    StackPlan p{};
    p.ok = false;
    if (M != 1 || d <= 0 || f <= 0 || (g != 64 && g != 128))
        return p;
    if (f % SGRID != 0 || (f / SX) % 32 != 0 || d % (SB * 8) != 0 || d % g != 0 || f % g != 0)
        return p;
    const int RG = f / SGRID, UG = d / 64, ng = d / g, UF = f / SX / 32, DJ = d / SB;
    if ((RG + 7) / 8 > SCW || ng % 4 != 0 || DJ > 128 || DJ % 16 != 0 || 2 * r + 1 > SPT)
        return p;
    if (r != 0 && r != 8 && r != 16 && r != 32)
        return p;
    if (UG % 8 != 0)                             // 8 lanes per row, no partial slot
        return p;
    p.jg = UG / 8;
    p.km = (4 * ng + 63) / 64;
    p.jd = (UF + 7) / 8;
    p.ndn = (DJ / 8 + SCW - 1) / SCW;
    if ((d / 16 + SPT - 1) / SPT > KXW || (f / SX / 8 + SPT - 1) / SPT > KHW)
        return p;
    if ((2 * r * (DJ / 8) + SCW * 64 - 1) / (SCW * 64) > KA)
        return p;
    const bool inst = (p.jg == 5 && p.km == 2 && p.jd == 5 && p.ndn == 2) ||
                      (p.jg == 8 && p.km == 2 && p.jd == 6 && p.ndn == 3) ||
                      (p.jg == 1 && p.km == 1 && p.jd == 1 && p.ndn == 1);
    if (!inst)
        return p;
    if (stack_cu_count() != SGRID)
        return p;
    size_t o = 16;
    auto take = [&](size_t bytes) { const size_t at = o; o = (o + bytes + 15) / 16 * 16; return (int)at; };
    p.o_xs = take((size_t)UG * 8 * 16);
    p.o_cx = take((size_t)UG * 8);
    p.o_t = take((size_t)(2 * r + 1) * 4);
    p.o_hs = take((size_t)p.jd * 8 * 4 * 16);     // chunk stride 8 JD >= UF units
    p.o_hcx = take((size_t)p.jd * 8 * 8);
    p.o_a = take((size_t)2 * r * DJ * 2 + 16);
    p.o_y = take((size_t)DJ * 2);
    p.o_xn = take((size_t)DJ * 2);
    p.meta_bytes = 2 * 8 * ng * 4 + 32 * r;      // metadata, then LoRA-B rows
    p.o_meta = take((size_t)SCW * p.meta_bytes);
    p.lds = o;
    p.ok = p.lds <= 64 * 1024;
    return p;
}

}  // namespace

bool stack_supported(int M, int d, int f, int g, int r) { return plan_stack(M, d, f, g, r).ok; }

size_t stack_ws_bytes(int d, int f, int r) {
    const size_t xw = (size_t)d + d / 4 + 2 * (2 * (size_t)r + 1) * SB;
    return 1024 + ((SX * xw * 4 + 255) & ~(size_t)255) + (((size_t)f * 4 + 255) & ~(size_t)255) +
           (size_t)2 * SX * d * 8;
}

int stack_max_layers() { return kStackMaxLayers; }

size_t stack_error_word_offset() { return (size_t)C_ERR * sizeof(unsigned); }

hipError_t launch_rmsnorm(const uint16_t* x, uint16_t* u, int M, int d, hipStream_t st) {
    if (M <= 0)
        return hipSuccess;
    rmsnorm_kernel<<<M, 256, 0, st>>>(x, u, d);
    return hipGetLastError();
}

hipError_t launch_residual(const uint16_t* x, const uint16_t* y, uint16_t* out, int n, bool bf16,
                           hipStream_t st) {
    if (n <= 0)
        return hipSuccess;
    residual_kernel<<<(n + 255) / 256, 256, 0, st>>>(x, y, out, n, bf16 ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_stack(const StackLayerDesc* layers, int L, int d, int f, int g, int r,
                        const uint16_t* x0, uint16_t* y, uint16_t* x_last, void* ws, hipStream_t st) {
    const StackPlan p = plan_stack(1, d, f, g, r);
    if (!p.ok || L <= 0 || L > kStackMaxLayers)
        return hipErrorInvalidValue;
    StackArgs a{};
    for (int i = 0; i < L; ++i) {
        const StackLayerDesc& s = layers[i];
        a.lay[i] = StackLayer{s.cg, s.mg, s.cu, s.mu, s.cd, s.md, s.Bg, s.Bu, s.Ag, s.Au, s.lora_scale};
    }
    a.L = L;
    a.d = d;
    a.f = f;
    a.g = g;
    a.r = r;
    a.x0 = x0;
    a.y = y;
    a.xl = x_last;
    char* base = static_cast<char*>(ws);
    a.ctl = reinterpret_cast<unsigned*>(base);
    const size_t xw = (size_t)d + d / 4 + 2 * (2 * (size_t)r + 1) * SB;
    a.xw = (int)xw;
    a.xb = reinterpret_cast<uint32_t*>(base + 1024);
    const size_t xbytes = (SX * xw * 4 + 255) & ~(size_t)255;
    a.hb = reinterpret_cast<uint32_t*>(base + 1024 + xbytes);
    a.pb = reinterpret_cast<unsigned long long*>(base + 1024 + xbytes + (((size_t)f * 4 + 255) & ~(size_t)255));
    a.o_xs = p.o_xs; a.o_cx = p.o_cx; a.o_t = p.o_t; a.o_hs = p.o_hs; a.o_hcx = p.o_hcx;
    a.o_a = p.o_a; a.o_y = p.o_y; a.o_xn = p.o_xn; a.o_meta = p.o_meta; a.meta_bytes = p.meta_bytes;
    auto run = [&](auto kernel) -> hipError_t {
        kernel<<<SGRID, STHREADS, p.lds, st>>>(a);
        return hipGetLastError();
    };
    if (p.jg == 5)
        return run(stack_kernel<5, 2, 5, 2>);
    if (p.jg == 8)
        return run(stack_kernel<8, 2, 6, 3>);
    return run(stack_kernel<1, 1, 1, 1>);
}

}  // namespace qmlp

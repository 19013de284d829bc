// Decode at several tokens (3 <= M <= 16, binary16) on the matrix cores,
// gfx950: a batch of independent blocks as two persistent launches after the
// LoRA-A products,
//
//   gate/up launch:  h_l = SiLU(W2gate x_l + s B_g t_g) * (W2up x_l + s B_u t_u)
//                    (Sec. 3.1 Eq. (1), Sec. 3.3, Sec. 4.2);
//   down launch:     y_l = W4down h_l (Sec. 3.3).
//
// With M tokens a weight feeds M multiply-adds; on the vector ALU that is
// M/2 dot2 operations per weight on top of its dequantization, more than the
// weight stream allows from a few tokens on.  Here every weight is unpacked
// once and multiplied into all tokens at once by v_mfma_f32_16x16x32_f16:
// the activation is the A operand (tokens as the 16 rows, padded), the codes
// the B operand (16 weight rows), D[token][weight row] in fp32.  A lane of a
// 16x16x32 step holds row (lane & 15) of each operand and K elements
// 8 (lane >> 4) .. + 7, and receives D rows 4 (lane >> 4) + v, column
// (lane & 15): the D values of a lane belong to its own weight row.
//
// Every MFMA step stays inside one quantization group, so the group's scale
// and zero apply exactly afterwards: lane quarter q = lane >> 4 covers a
// fixed set of 16-code (2-bit) or 8-code (4-bit) words of each group.  The
// codes enter as in the other decode kernels: a field OR-ed into binary16
// 1024.0 reads 1024 + c 2^j, the activation is staged pre-scaled by 2^-j in
// the same pair order per word, and each group's accumulator starts at
// -(C + z X) (C = 1024 sum x', X = sum x per token and group), so the group
// adds s * acc.  The LoRA-B term is one more MFMA per item: lora_scale * t
// (binary16, zero past the rank) times the item's B rows.
//
// Loads.  Every code load is 16 bytes per lane and fetches eight weight
// rows' 128-byte lines whole; the words then move between lanes in
// registers (a row rotation, v_permlane16_swap, v_permlane32_swap) so that
// lane 16 q + j holds row j and each quarter q words of every group (see
// "Whole-line loads" below).
//
// Work split.  Each workgroup owns a contiguous range of the batch's
// 16-row items (flattened over blocks).
//   gate/up: the whole x' of the block an item belongs to sits in LDS (MT
//     token rows, MT = 4, 8 or 16 >= M; A rows past MT re-read token
//     row & (MT - 1), their results are never stored); a range touching two
//     blocks stages them one after the other.  Waves take the range's items
//     in turn and stream each item's codes in steps of four groups with two
//     register sets.
//   down: h' of a block is too large for LDS at these widths, so the K
//     dimension (f) is walked in steps of two groups: every wave keeps the
//     accumulators of its few items for the whole walk, and h' is staged in
//     chunks of several steps into two LDS buffers that all waves share (one
//     barrier per chunk).
#include "decode_common.h"
#include "decode_launch.h"

namespace qmlp {

namespace {

typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef const BatchArgs __attribute__((address_space(4))) KBatchM;
__device__ __forceinline__ KBatchM* kbm() { return (KBatchM*)__builtin_amdgcn_kernarg_segment_ptr(); }

__device__ __forceinline__ f32x4_t mfma16(const uint4& a, const uint4& b, f32x4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                  __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

// Lanes 32-63 of a trade places with lanes 0-31 of b.
__device__ __forceinline__ void swap32(uint32_t& a, uint32_t& b) {
    const auto r = __builtin_amdgcn_permlane32_swap(a, b, false, false);
    a = r[0];
    b = r[1];
}
// Lanes 16-31 and 48-63 of a trade places with lanes 0-15 and 32-47 of b.
__device__ __forceinline__ void swap16(uint32_t& a, uint32_t& b) {
    const auto r = __builtin_amdgcn_permlane16_swap(a, b, false, false);
    a = r[0];
    b = r[1];
}

// LDS barrier that leaves vector-memory loads in flight: this wave's LDS
// accesses complete, then the workgroup meets.
__device__ __forceinline__ void lds_barrier() {
    __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Weight loads go through buffer resources: a resource of zero bytes turns
// a load into one that returns zeros without touching memory, so a prefetch
// that has nothing to fetch issues the same instructions as one that has
// (the compiler then keeps the next step's loads in flight across a step),
// and every load is bounds-checked against its array.
typedef __amdgpu_buffer_rsrc_t Rsrc;
__device__ __forceinline__ Rsrc rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
constexpr int kAuxNt = 2;      // non-temporal: codes are read once
template <int AUX>
__device__ __forceinline__ uint4 bload16(Rsrc r, uint32_t voff, uint32_t soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, AUX);
    return make_uint4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ uint2 bload8(Rsrc r, uint32_t voff, uint32_t soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0);
    return make_uint2(v[0], v[1]);
}

constexpr int kMfWaves = 12;   // waves per workgroup (one workgroup per compute unit)

// Whole-line loads.  A step reads 128 bytes (eight 16-byte units) of each of
// 16 weight rows; each load instruction covers 8 rows whole (lane L: row
// 8 h + (L & 7) for load h, unit u(L) from lane bits 5..3), so every 128-byte
// line is fetched by one instruction.  The matrix cores want lane l = 16 q + j
// to hold row j, so the units are then moved between lanes in registers: with
// the row bit h exchanged for lane bit 3 (E3, a row rotation by 8 under a
// bank mask), the 4-byte words of a unit u = (u2 u1 u0), w = (w1 w0) sit at
// register (u2 after E3) and component (w1 w0); E4 exchanges lane bit 4 with
// component bit w1 (v_permlane16_swap) and E5 lane bit 5 with w0
// (v_permlane32_swap).  Which unit bit each lane bit carries is chosen per
// layout so that a quarter's words of one group end up in the same register
// positions for every group (QW words per quarter and group):
//   2-bit g = 128, 4-bit g = 64 (E3, E4): lane bits 5, 4, 3 = u0, u1, u2;
//     quarter q holds words 2q, 2q + 1 of a group;
//   2-bit g = 64 (E3, E4, E5): same units; quarter q holds word
//     2 (q & 1) + (q >> 1) of each group;
//   4-bit g = 128 (E3): lane bits 5, 4, 3 = u1, u0, u2; quarter q holds
//     words 4q .. 4q + 3.
template <int QW>
__device__ __forceinline__ int quarter_word(int q) {
    if constexpr (QW == 1) return 2 * (q & 1) + (q >> 1);
    else if constexpr (QW == 2) return 2 * q;
    else return 4 * q;
}
// 16-byte unit of the step's 128 bytes that lane L loads.
template <bool DN128>
__device__ __forceinline__ int lane_unit(int L) {
    const int b5 = (L >> 5) & 1, b4 = (L >> 4) & 1, b3 = (L >> 3) & 1;
    return DN128 ? 4 * b3 + 2 * b5 + b4 : 4 * b3 + 2 * b4 + b5;
}
constexpr int kDppRowRor8 = 0x128;
// E3 on one component: a (h = 0) and b (h = 1) become the S3 = 0 and S3 = 1
// halves, rows 8..15 taken from lane l ^ 8.
__device__ __forceinline__ void e3(uint32_t& a, uint32_t& b) {
    const int na = __builtin_amdgcn_update_dpp((int)a, (int)b, kDppRowRor8, 0xF, 0xC, false);
    const int nb = __builtin_amdgcn_update_dpp((int)b, (int)a, kDppRowRor8, 0xF, 0x3, false);
    a = (uint32_t)na;
    b = (uint32_t)nb;
}
// The exchanges of a step's two loads: E3 always, E4 and E5 as asked.
template <bool E4, bool E5>
__device__ __forceinline__ void arrange(uint4 (&v)[2]) {
    e3(v[0].x, v[1].x);
    e3(v[0].y, v[1].y);
    e3(v[0].z, v[1].z);
    e3(v[0].w, v[1].w);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        if constexpr (E4) {
            swap16(v[i].x, v[i].z);
            swap16(v[i].y, v[i].w);
        }
        if constexpr (E5) {
            swap32(v[i].x, v[i].y);
            swap32(v[i].z, v[i].w);
        }
    }
}

// ---------------------------------------------------------------- staging
// Staging word W (16 values) of token j of an activation into x' halves
// (pairs (x[p], x[8 + p]), pre-scaled; layout [W][half][MT] with one pad
// entry per word, so that the lanes writing consecutive words hit distinct
// LDS banks) and the
// (-C, -X) of its group (GW words per group on GW consecutive lanes; every
// lane of the wave calls this).
template <int MT, int GW>
__device__ __forceinline__ void mf_stage_word(uint4* xs, float2* cx, int W, int j, bool live, const uint4& lo16,
                                              const uint4& hi16) {
    const uint32_t xl[4] = {lo16.x, lo16.y, lo16.z, lo16.w};
    const uint32_t xh[4] = {hi16.x, hi16.y, hi16.z, hi16.w};
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
    csum = group_sum<GW>(csum);
    xsum = group_sum<GW>(xsum);
    if (live) {
        xs[W * (2 * MT + 1) + j] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        xs[W * (2 * MT + 1) + MT + j] = make_uint4(pr[4], pr[5], pr[6], pr[7]);
        if (W % GW == 0)
            cx[(W / GW) * MT + j] = make_float2(-1024.0f * csum, -xsum);
    }
}

// 4-bit words: 8 values of token j (one 16-byte load) as pairs (h[p], h[4 + p])
// pre-scaled for the positions {0, 4, 0, 4}; layout [W][MT + 1] (the pad makes
// the 16 lanes that write consecutive words of one token hit distinct LDS
// banks); GW words per group.
template <int MT, int GW>
__device__ __forceinline__ void mf_stage_word4(uint4* hs, float2* cx, int W, int j, bool live, const uint4& v) {
    const uint32_t hl[4] = {v.x, v.y, v.z, v.w};
    uint32_t pr[4];
    float csum = 0.0f, xsum = 0.0f;
#pragma unroll
    for (int p = 0; p < 4; ++p) {
        const uint32_t a16 = (hl[p >> 1] >> (16 * (p & 1))) & 0xFFFFu;
        const uint32_t b16 = (hl[2 + (p >> 1)] >> (16 * (p & 1))) & 0xFFFFu;
        const float sc = w4_s1_scale(p);
        const uint32_t ha = f2h(h2f(a16) * sc), hb = f2h(h2f(b16) * sc);
        pr[p] = ha | (hb << 16);
        csum += h2f(ha) + h2f(hb);
        xsum += h2f(a16) + h2f(b16);
    }
    csum = group_sum<GW>(csum);
    xsum = group_sum<GW>(xsum);
    if (live) {
        hs[W * (MT + 1) + j] = make_uint4(pr[0], pr[1], pr[2], pr[3]);
        if (W % GW == 0)
            cx[(W / GW) * MT + j] = make_float2(-1024.0f * csum, -xsum);
    }
}

// ---------------------------------------------------------------- gate/up
// One step of an item: 128 bytes of each of its 16 rows per matrix (512
// codes, GSU = 512 / G groups) in two loads, and the rows' (scale | zero)
// words of those groups (MW = GSU / 4 loads).
template <int G>
struct MfGuBuf {
    static constexpr int GSU = 512 / G, MW = GSU / 4;
    uint4 cg[2], cu[2];
    uint4 mg[MW], mu[MW];
    uint4 bg, bu;            // LoRA-B ranks 8 q .. 8 q + 7 of the row (last step of an item)
};

__device__ __forceinline__ uint32_t word_of(const uint4& v, int i) {
    return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// Step c of the item whose first row is row n of block l: the two
// whole-line loads per matrix (rows n + 8 i + (lane & 7)), and for lane row
// n + (lane & 15) its (scale | zero) words and LoRA-B ranks.  A prefetch
// past a wave's last step (dummy), and the LoRA-B rows on every step but an
// item's last, load from empty resources.  The (scale | zero) words are
// plain loads: a row's line of them serves several steps.
template <int G>
__device__ __forceinline__ void mf_gu_load(MfGuBuf<G>& q, int l, int n, int c, int nsb, int d, int f, int r,
                                           bool dummy, int lane) {
    constexpr int GSU = 512 / G, MW = GSU / 4;
    KBatchM* kb = kbm();
    const int qt = lane >> 4, lr = lane & 15;
    const int ng = d / G, rw = d / 16;
    const uint32_t cbytes = dummy ? 0u : (uint32_t)f * (uint32_t)(d / 4);
    const uint32_t mbytes = dummy ? 0u : (uint32_t)f * (uint32_t)ng * 4u;
    const Rsrc rg = rsrc(kb->lay[l].cg, cbytes), ru = rsrc(kb->lay[l].cu, cbytes);
    const Rsrc sg = rsrc(kb->lay[l].mg, mbytes), su = rsrc(kb->lay[l].mu, mbytes);
    const uint32_t cv = (uint32_t)((lane & 7) * rw) * 4u + 16u * (uint32_t)lane_unit<false>(lane);
    const uint32_t cs = (uint32_t)(n * rw + c * 32) * 4u;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        q.cg[i] = bload16<kAuxNt>(rg, cv + (uint32_t)(8 * i * rw) * 4u, cs);
        q.cu[i] = bload16<kAuxNt>(ru, cv + (uint32_t)(8 * i * rw) * 4u, cs);
    }
    const uint32_t mv = (uint32_t)(lr * ng) * 4u, ms = (uint32_t)(n * ng + c * GSU) * 4u;
#pragma unroll
    for (int i = 0; i < MW; ++i) {
        q.mg[i] = bload16<0>(sg, mv + 16 * i, ms);
        q.mu[i] = bload16<0>(su, mv + 16 * i, ms);
    }
    const bool lora = !dummy && c == nsb - 1 && r > 0;
    const uint32_t bbytes = lora ? (uint32_t)f * (uint32_t)r * 2u : 0u;
    const Rsrc bg = rsrc(kb->lay[l].Bg, bbytes), bu = rsrc(kb->lay[l].Bu, bbytes);
    const uint32_t bv = (uint32_t)(lr * r + (8 * qt < r ? 8 * qt : 0)) * 2u, bs = (uint32_t)(n * r) * 2u;
    q.bg = bload16<0>(bg, bv, bs);
    q.bu = bload16<0>(bu, bv, bs);
}

// Words of group i (0 .. GSU - 1) of the step for this lane (QW = G / 64
// each) from the arranged loads.
template <int G>
__device__ __forceinline__ void mf_gu_words(uint4 (&v)[2], uint32_t (&w)[512 / G][G / 64]) {
    arrange<true, G == 64>(v);
#pragma unroll
    for (int g = 0; g < 512 / G; ++g) {
        if constexpr (G == 64)
            w[g][0] = word_of(v[g >> 2], g & 3);
        else {
            w[g][0] = word_of(v[g >> 1], 2 * (g & 1));
            w[g][1] = word_of(v[g >> 1], 2 * (g & 1) + 1);
        }
    }
}

template <int G, int MT>
__device__ __forceinline__ void mf_gu_step(MfGuBuf<G>& q, const uint4* xsb, const float2* cxb, int c, int lane,
                                           f32x4_t& G4, f32x4_t& U4) {
    constexpr int QW = G / 64, WPG = G / 16, GSU = 512 / G;
    const uint32_t mv = magic_vgpr();
    const int qt = lane >> 4;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        pin4(q.cg[i]);
        pin4(q.cu[i]);
    }
    uint32_t wg[GSU][QW], wu[GSU][QW];
    mf_gu_words<G>(q.cg, wg);
    mf_gu_words<G>(q.cu, wu);
#pragma unroll
    for (int i = 0; i < GSU; ++i) {
        const int t = c * GSU + i;
        const uint32_t mgi = word_of(q.mg[i / 4], i % 4), mui = word_of(q.mu[i / 4], i % 4);
        // (-C, -X) of the tokens of this lane's D rows, 4 (q & (MT/4 - 1)) .. + 3
        const float2* cl = cxb + t * MT + 4 * (qt & (MT / 4 - 1));
        const float2 k0 = cl[0], k1 = cl[1], k2 = cl[2], k3 = cl[3];
        const float zg = h2f(mgi >> 16), zu = h2f(mui >> 16);
        f32x4_t ag = {zg * k0.y + k0.x, zg * k1.y + k1.x, zg * k2.y + k2.x, zg * k3.y + k3.x};
        f32x4_t au = {zu * k0.y + k0.x, zu * k1.y + k1.x, zu * k2.y + k2.x, zu * k3.y + k3.x};
#pragma unroll
        for (int w = 0; w < QW; ++w) {
            uint32_t eg[8], eu[8];
            extract_w2_s1(wg[i][w], eg, mv);
            extract_w2_s1(wu[i][w], eu, mv);
            const int W = t * WPG + w;                         // plus the lane's quarter offset (in xsb)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const uint4 a = xsb[W * (2 * MT + 1) + h * MT];
                ag = mfma16(a, make_uint4(eg[4 * h], eg[4 * h + 1], eg[4 * h + 2], eg[4 * h + 3]), ag);
                au = mfma16(a, make_uint4(eu[4 * h], eu[4 * h + 1], eu[4 * h + 2], eu[4 * h + 3]), au);
            }
        }
        G4 += h2f(mgi & 0xFFFFu) * ag;
        U4 += h2f(mui & 0xFFFFu) * au;
    }
}

// ---------------------------------------------------------------- LoRA-A
// t = [A_g; A_u] x of every block of the batch (Sec. 3.1 Eq. (1), Sec. 4.2),
// also on the matrix cores: workgroup (tile, slice) of block l multiplies 16
// rows of [A_g; A_u] (rows past r are those of A_u) by the block's tokens
// over slice s of d (the tokens as the A operand, padded with token 0 whose
// results are dropped).  Its four waves take a quarter of the slice each
// and add their sums in wave order through LDS; the fp32 partial goes to
// t[s][l][token][row] and the gate/up launch adds the kLoraSlices partials
// in slice order.  Every wave streams 16 rows x 64 bytes per load from
// independent addresses, so nothing here waits on another workgroup.
__global__ void __launch_bounds__(256) mf_lora_kernel(BatchArgs b, int nb) {
    __shared__ float red[4][4][64];                       // [wave][v][lane]
    const int l = blockIdx.y;
    const int tile = blockIdx.x / kLoraSlices, s = blockIdx.x - tile * kLoraSlices;
    const int d = b.d, r = b.r, M = b.M;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, q = lane >> 4;
    const int c = tile * 16 + (lane & 15);                // this lane's row of [A_g; A_u]
    const int kc = d / (4 * kLoraSlices);                 // K of one wave, a multiple of 32
    const int nst = kc / 32;
    const int k0 = (s * 4 + wave) * kc + 8 * q;
    const uint16_t* ar = c < r ? kbm()->lay[l].Ag + (long)c * d : kbm()->lay[l].Au + (long)(c - r) * d;
    const int j = (lane & 15) < M ? (lane & 15) : 0;
    const uint16_t* xr = b.x + ((long)l * M + j) * d;
    f32x4_t acc = {0.0f, 0.0f, 0.0f, 0.0f};
    constexpr int KC = 4;                                 // steps whose loads go out together
    for (int i = 0; i < nst; i += KC) {
        uint4 av[KC], xv[KC];
#pragma unroll
        for (int u = 0; u < KC; ++u) {
            const int k = k0 + 32 * (i + u < nst ? i + u : nst - 1);
            av[u] = *reinterpret_cast<const uint4*>(ar + k);
            xv[u] = *reinterpret_cast<const uint4*>(xr + k);
        }
#pragma unroll
        for (int u = 0; u < KC; ++u)
            if (i + u < nst)
                acc = mfma16(xv[u], av[u], acc);
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) red[wave][v][lane] = acc[v];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float sum = ((red[0][v][lane] + red[1][v][lane]) + red[2][v][lane]) + red[3][v][lane];
            const int tok = 4 * q + v;                    // D row of this lane and v
            if (tok < M)
                b.t[(((long)s * nb + l) * M + tok) * 2 * r + c] = sum;
        }
    }
}

template <int G, int MT, int NW>
__global__ void __launch_bounds__(NW * 64) mf_gu_kernel(BatchArgs b, int nb) {
    constexpr int NT = NW * 64, GW = G / 16, QW = G / 64;
    const int d = b.d, f = b.f, r = b.r, M = b.M;
    const int nsb = d / 512;                              // steps per item
    const int NWd = d / 16;                               // 16-code words per row
    extern __shared__ uint4 smem[];
    uint4* xs = smem;                                                    // [NWd][2 MT + 1]
    float2* cx = reinterpret_cast<float2*>(smem + NWd * (2 * MT + 1));    // [d/G][MT]
    uint16_t* tsg = reinterpret_cast<uint16_t*>(cx + (d / G) * MT);       // [MT][32] lora_scale t_g
    uint16_t* tsu = tsg + MT * 32;                                       // [MT][32] lora_scale t_u
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ipb = f / 16;                               // items per block
    const int qt = lane >> 4, jj = (lane & 15) & (MT - 1);

    const int nit = nb * ipb;
    const int i0 = (int)((long)blockIdx.x * nit / gridDim.x), i1 = (int)((long)(blockIdx.x + 1) * nit / gridDim.x);
    for (int seg = i0; seg < i1;) {
        const int l = seg / ipb;
        const int send = (l + 1) * ipb < i1 ? (l + 1) * ipb : i1;
        // ---- stage x' of block l, its (-C, -X) and lora_scale * t
        __syncthreads();                                  // the previous segment is done with LDS
        {
            const uint16_t* xl = b.x + (long)l * M * d;
            const int words = MT * NWd;
            for (int idx = tid; idx < ((words + 63) & ~63); idx += NT) {
                const bool live = idx < words;
                const int j = live ? idx / NWd : 0, W = live ? idx - j * NWd : 0;
                const bool data = live && j < M;
                const uint4* src = reinterpret_cast<const uint4*>(xl + (long)(data ? j : 0) * d) + 2 * W;
                uint4 lo = src[0], hi = src[1];
                if (!data)
                    lo = hi = make_uint4(0u, 0u, 0u, 0u);
                mf_stage_word<MT, GW>(xs, cx, W, j, live, lo, hi);
            }
            const float ls = kbm()->lay[l].lora_scale;
            for (int k = tid; k < MT * 32; k += NT) {
                const int j = k >> 5, c = k & 31;
                const bool ok = j < M && c < r;
                // the LoRA-A partials of the kLoraSlices slices of d, added in order
                const float* tl = b.t + ((long)l * M + (ok ? j : 0)) * 2 * r;
                const long ps = (long)nb * M * 2 * r;
                float vg = 0.0f, vu = 0.0f;
                if (ok) {
#pragma unroll
                    for (int sl = 0; sl < kLoraSlices; ++sl) {
                        vg += tl[sl * ps + c];
                        vu += tl[sl * ps + r + c];
                    }
                }
                tsg[k] = (uint16_t)f2h(ls * vg);
                tsu[k] = (uint16_t)f2h(ls * vu);
            }
        }
        __syncthreads();
        // ---- this wave's items of the segment, nsb steps each, two register sets
        const int first = seg + wave;
        const int nk = first < send ? (send - first + NW - 1) / NW : 0;
        const int nsteps = nk * nsb;
        if (nsteps > 0) {
            const uint4* xsb = xs + quarter_word<QW>(qt) * (2 * MT + 1) + jj;   // this lane's A base
            int ld_item = first, ld_c = 0, left = nsteps - 1;
            int cp_item = first, cp_c = 0;
            auto advance = [&]() {
                if (left > 0) {
                    --left;
                    if (++ld_c == nsb) {
                        ld_c = 0;
                        ld_item += NW;
                    }
                    return true;
                }
                return false;
            };
            MfGuBuf<G> A, B;
            mf_gu_load<G>(A, l, (ld_item - l * ipb) * 16, ld_c, nsb, d, f, r, false, lane);
            f32x4_t Gt = {0.f, 0.f, 0.f, 0.f}, Ut = {0.f, 0.f, 0.f, 0.f};
            auto run = [&](MfGuBuf<G>& q) {
                mf_gu_step<G, MT>(q, xsb, cx, cp_c, lane, Gt, Ut);
                if (cp_c == nsb - 1) {
                    if (r > 0) {
                        // LoRA-B: lora_scale * t (A rows = tokens) times the item's B rows
                        const uint4 ag = *reinterpret_cast<const uint4*>(tsg + jj * 32 + 8 * qt);
                        const uint4 au = *reinterpret_cast<const uint4*>(tsu + jj * 32 + 8 * qt);
                        Gt = mfma16(ag, q.bg, Gt);
                        Ut = mfma16(au, q.bu, Ut);
                    }
                    const int n = (cp_item - l * ipb) * 16 + (lane & 15);
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int tok = 4 * qt + v;
                        const float gv = Gt[v], uv = Ut[v];
                        if (tok < M)
                            b.h[((long)l * M + tok) * f + n] = (uint16_t)f2h(gv / (1.0f + __expf(-gv)) * uv);
                    }
                    Gt = f32x4_t{0.f, 0.f, 0.f, 0.f};
                    Ut = f32x4_t{0.f, 0.f, 0.f, 0.f};
                    cp_c = 0;
                    cp_item += NW;
                } else {
                    ++cp_c;
                }
            };
            for (int st = 0; st < nsteps; st += 2) {
                bool real = advance();
                mf_gu_load<G>(B, l, (ld_item - l * ipb) * 16, ld_c, nsb, d, f, r, !real, lane);
                run(A);
                real = advance();
                mf_gu_load<G>(A, l, (ld_item - l * ipb) * 16, ld_c, nsb, d, f, r, !real, lane);
                if (st + 1 < nsteps)
                    run(B);
            }
        }
        seg = send;
    }
}

// ---------------------------------------------------------------- down
// One step of TPW items: 128 bytes of each row (256 codes, GSD = 256 / G
// groups) in two loads per item, and the rows' (scale | zero) words of those
// groups.
template <int G>
struct MfDnMeta;
template <>
struct MfDnMeta<128> {
    typedef uint2 type;       // two groups
};
template <>
struct MfDnMeta<64> {
    typedef uint4 type;       // four groups
};
template <int G, int TPW>
struct MfDnBuf {
    uint4 c[TPW][2];
    typename MfDnMeta<G>::type m[TPW];
};

__device__ __forceinline__ uint32_t word_of(const uint2& v, int i) { return i == 0 ? v.x : v.y; }

// Step k of the wave's items: item tt has its first row at row0 + tt * srow;
// its two whole-line loads cover rows + 8 i + (lane & 7), its (scale | zero)
// words are lane row + (lane & 15)'s.  Items at or past ntile, and a
// prefetch past the last step, load from empty resources.
template <int G, int TPW>
__device__ __forceinline__ void mf_dn_load(MfDnBuf<G, TPW>& q, int l, int row0, int srow, int ntile, int k, int d,
                                           int f, bool dummy, int lane) {
    constexpr int GSD = 256 / G;
    KBatchM* kb = kbm();
    const int lr = lane & 15, ng = f / G, rw = f / 8;
    const uint32_t cv = (uint32_t)((lane & 7) * rw) * 4u + 16u * (uint32_t)lane_unit<G == 128>(lane);
    const uint32_t mv = (uint32_t)(lr * ng) * 4u;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
        const bool real = !dummy && tt < ntile;
        const Rsrc rc = rsrc(kb->lay[l].cd, real ? (uint32_t)d * (uint32_t)(f / 2) : 0u);
        const Rsrc rm = rsrc(kb->lay[l].md, real ? (uint32_t)d * (uint32_t)ng * 4u : 0u);
        const int row = row0 + tt * srow;
        const uint32_t cs = (uint32_t)(row * rw + k * 32) * 4u, ms = (uint32_t)(row * ng + k * GSD) * 4u;
#pragma unroll
        for (int i = 0; i < 2; ++i) q.c[tt][i] = bload16<kAuxNt>(rc, cv + (uint32_t)(8 * i * rw) * 4u, cs);
        if constexpr (G == 128)
            q.m[tt] = bload8(rm, mv, ms);
        else
            q.m[tt] = bload16<0>(rm, mv, ms);
    }
}

// Word ww (0 .. G/32 - 1) of group i (0 .. GSD - 1) of the step for this
// lane, from the item's loads after mf_dn_arrange: g = 128, register i,
// components ww; g = 64, register i >> 1, components 2 (i & 1) + ww.
template <int G>
__device__ __forceinline__ uint32_t mf_dn_word(const uint4 (&v)[2], int i, int ww) {
    if constexpr (G == 128)
        return word_of(v[i], ww);
    else
        return word_of(v[i >> 1], 2 * (i & 1) + ww);
}
template <int G>
__device__ __forceinline__ void mf_dn_arrange(uint4 (&v)[2]) {
    arrange<G == 64, false>(v);
}

template <int G, int MT, int TPW>
__device__ __forceinline__ void mf_dn_step(MfDnBuf<G, TPW>& q, const uint4* hsb, const float2* cxb, int ntile,
                                           int lane, f32x4_t (&Y)[TPW]) {
    constexpr int QW = G / 32, WPG = G / 8, GSD = 256 / G;
    const uint32_t mv = magic_vgpr();
    const int qt = lane >> 4;
#pragma unroll
    for (int tt = 0; tt < TPW; ++tt) {
        if (tt < ntile) {
            pin4(q.c[tt][0]);
            pin4(q.c[tt][1]);
            mf_dn_arrange<G>(q.c[tt]);
        }
    }
#pragma unroll
    for (int i = 0; i < GSD; ++i) {
        const float2* cl = cxb + i * MT + 4 * (qt & (MT / 4 - 1));
        const float2 k0 = cl[0], k1 = cl[1], k2 = cl[2], k3 = cl[3];
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt) {
            if (tt < ntile) {
                const uint32_t mw = word_of(q.m[tt], i);
                const float z = h2f(mw >> 16);
                f32x4_t acc = {z * k0.y + k0.x, z * k1.y + k1.x, z * k2.y + k2.x, z * k3.y + k3.x};
#pragma unroll
                for (int ww = 0; ww < QW; ++ww) {
                    uint32_t e[4];
                    extract_w4_s1(mf_dn_word<G>(q.c[tt], i, ww), e, mv);
                    acc = mfma16(hsb[(i * WPG + ww) * (MT + 1)], make_uint4(e[0], e[1], e[2], e[3]), acc);
                }
                Y[tt] += h2f(mw & 0xFFFFu) * acc;
            }
        }
    }
}

// h' staging: each thread holds SPT 16-byte words of a chunk between
// issuing their loads and writing them to LDS.
template <int SPT>
struct MfStage {
    uint4 v[SPT];
};

// ck: codes of f per staged chunk (a multiple of 256, with MT ck / 8 <= SPT NT).
template <int G, int MT, int TPW, int NW, int SPT>
__global__ void __launch_bounds__(NW * 64) mf_dn_kernel(BatchArgs b, int nb, int ck) {
    constexpr int NT = NW * 64, GW = G / 8, QW = G / 32;
    const int d = b.d, f = b.f, M = b.M;
    const int nsteps = f / 256;
    const int sc = ck / 256;                              // steps per chunk
    const int nchunk = (nsteps + sc - 1) / sc;
    const int ckw = ck / 8, ckg = ck / G;                 // words and groups per chunk row
    extern __shared__ uint4 smem[];
    uint4* hs = smem;                                                     // [2][ckw][MT + 1]
    float2* cx = reinterpret_cast<float2*>(smem + 2 * ckw * (MT + 1));    // [2][ckg][MT]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ipb = d / 16;
    const int qt = lane >> 4, jj = (lane & 15) & (MT - 1);
    const int qoff = quarter_word<QW>(qt) * (MT + 1) + jj;

    const int nit = nb * ipb;
    const int i0 = (int)((long)blockIdx.x * nit / gridDim.x), i1 = (int)((long)(blockIdx.x + 1) * nit / gridDim.x);
    MfStage<SPT> sb;
    // this thread's staging words of a chunk: word sW of token sj (sj >= MT:
    // past the chunk)
    int sj[SPT], sW[SPT];
#pragma unroll
    for (int s = 0; s < SPT; ++s) {
        const int idx = tid + s * NT;
        sj[s] = idx / ckw;
        sW[s] = idx - sj[s] * ckw;
    }
    // Segments: the range's items of one block, in rounds of at most TPW
    // items per wave, each round a full walk over f.
    for (int seg = i0; seg < i1;) {
        const int l = seg / ipb;
        const int bend = (l + 1) * ipb < i1 ? (l + 1) * ipb : i1;
        const int rounds = (bend - seg + TPW * NW - 1) / (TPW * NW);
        const int send = seg + (bend - seg + rounds - 1) / rounds;
        const int first = seg + wave;
        const int ntile = first < send ? (send - first + NW - 1) / NW : 0;     // <= TPW
        // h' of chunk c: thread word s is word sW[s] of token sj[s]; padding
        // tokens and words past a short last chunk load from outside the
        // resource (zeros) and are dropped
        const Rsrc rh = rsrc(b.h + (long)l * M * f, (uint32_t)M * (uint32_t)f * 2u);
        auto chunk_words = [&](int c) { return ((c + 1) * ck <= f ? ck : f - c * ck) / 8; };
        auto stage_issue = [&](int c) {
            const int cw = chunk_words(c);
#pragma unroll
            for (int s = 0; s < SPT; ++s) {
                const bool data = sj[s] < M && sW[s] < cw;
                const uint32_t vo = data ? (uint32_t)(sj[s] * f + 8 * sW[s]) * 2u : 0x80000000u;
                sb.v[s] = bload16<0>(rh, vo, (uint32_t)(c * ck) * 2u);
            }
        };
        auto stage_commit = [&](int c) {
            uint4* hb = hs + (c & 1) * ckw * (MT + 1);
            float2* cb = cx + (c & 1) * ckg * MT;
            const int cw = chunk_words(c);
#pragma unroll
            for (int s = 0; s < SPT; ++s)
                if (s * NT < MT * ckw)                    // uniform: the workgroup's last words
                    mf_stage_word4<MT, GW>(hb, cb, sW[s], sj[s], sj[s] < MT && sW[s] < cw, sb.v[s]);
        };
        lds_barrier();                                     // the previous round is done with LDS
        stage_issue(0);
        stage_commit(0);
        f32x4_t Y[TPW];
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt) Y[tt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
        const int row0 = (first - l * ipb) * 16;
        MfDnBuf<G, TPW> A, B;
        mf_dn_load<G, TPW>(A, l, row0, 16 * NW, ntile, 0, d, f, false, lane);
        int kin = 0, cbuf = 0, cnext = 1;
        auto body = [&](MfDnBuf<G, TPW>& cur, MfDnBuf<G, TPW>& nxt, int k) {
            // at a chunk's first step: chunk cnext - 1 is in LDS (every wave
            // waited for its own writes) and chunk cnext - 2 is consumed, so
            // chunk cnext is loaded now (after the next step's prefetch) and
            // written after this step's work
            const bool stg = kin == 0 && cnext < nchunk;
            if (kin == 0)
                lds_barrier();
            const bool more = k + 1 < nsteps;
            mf_dn_load<G, TPW>(nxt, l, row0, 16 * NW, ntile, more ? k + 1 : k, d, f, !more, lane);
            if (stg)
                stage_issue(cnext);
            mf_dn_step<G, MT, TPW>(cur, hs + cbuf * ckw * (MT + 1) + kin * 32 * (MT + 1) + qoff,
                                   cx + cbuf * ckg * MT + kin * (256 / G) * MT, ntile, lane, Y);
            if (stg)
                stage_commit(cnext);
            if (kin == 0)
                ++cnext;
            if (++kin == sc) {
                kin = 0;
                cbuf ^= 1;
            }
        };
        for (int k = 0; k < nsteps; k += 2) {
            body(A, B, k);
            if (k + 1 < nsteps)
                body(B, A, k + 1);
        }
        // y of the wave's items: D[token 4 q + v][row lane & 15]
#pragma unroll
        for (int tt = 0; tt < TPW; ++tt) {
            if (tt < ntile) {
                const int o = row0 + tt * 16 * NW + (lane & 15);
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int tok = 4 * qt + v;
                    if (tok < M)
                        b.y[((long)l * M + tok) * d + o] = (uint16_t)f2h(Y[tt][v]);
                }
            }
        }
        seg = send;
    }
}

int mf_cu_count() {
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

constexpr size_t kMfLds = 160 * 1024;

int mf_mt(int M) { return M <= 4 ? 4 : M <= 8 ? 8 : 16; }

size_t mf_gu_lds(int d, int g, int MT) {
    return (size_t)(d / 16) * (2 * MT + 1) * 16 + (size_t)(d / g) * MT * 8 + 2 * MT * 32 * 2;
}
size_t mf_dn_lds(int ck, int g, int MT) {
    return (size_t)2 * (ck / 8) * (MT + 1) * 16 + (size_t)2 * (ck / g) * MT * 8;
}
// down: items per wave and round, and waves per workgroup, by token tile (at
// MT = 8 two items per wave measured 3 % faster on the 14B-class blocks than
// three; other choices, such as 8 waves of 4 items at MT = 4, stayed within
// the run-to-run spread)
constexpr int dn_tpw(int MT) { return MT == 8 ? 2 : 3; }
constexpr int dn_waves(int MT) { return kMfWaves; }
// down: staged h' words per thread and chunk (registers left beside the
// items' loads: those of g = 64 carry twice the (scale | zero) words)
constexpr int mf_stage_words(int g) { return g == 64 ? 2 : 4; }
// Codes per staged h' chunk: the largest multiple of 256 whose MT tokens fit
// the staging registers of the workgroup and whose two buffers fit in LDS,
// no larger than f rounded up to a step.
int mf_dn_chunk(int f, int g, int MT) {
    int ck = mf_stage_words(g) * dn_waves(MT) * 64 * 8 / MT / 256 * 256;
    while (ck > 256 && mf_dn_lds(ck, g, MT) > kMfLds) ck -= 256;
    const int fr = (f + 255) / 256 * 256;
    return ck < fr ? ck : fr;
}
int mf_grid(long items) {
    const long c = mf_cu_count();
    return (int)(items < c ? items : c);
}

}  // namespace

bool mfma_supported(int M, int d, int f, int gg, int bg, int gd, int bd, int r, int nb) {
    if (M < 3 || M > 16 || bg != 2 || bd != 4 || (gg != 64 && gg != 128) || (gd != 64 && gd != 128))
        return false;
    if (r != 0 && r != 8 && r != 16 && r != 32)
        return false;
    if (nb < 1 || nb > kBatchMax || d % 512 != 0 || f % 256 != 0)
        return false;
    if (mf_cu_count() <= 0)
        return false;
    const int MT = mf_mt(M);
    return mf_gu_lds(d, gg, MT) <= kMfLds && mf_dn_lds(mf_dn_chunk(f, gd, MT), gd, MT) <= kMfLds;
}

hipError_t launch_lora_a_mfma(const BatchArgs& b, int nb, hipStream_t st) {
    if (!mfma_supported(b.M, b.d, b.f, b.gg, b.bg, b.gd, b.bd, b.r, nb) || b.r == 0)
        return hipErrorInvalidValue;
    mf_lora_kernel<<<dim3((unsigned)(2 * b.r / 16 * kLoraSlices), (unsigned)nb), 256, 0, st>>>(b, nb);
    return hipGetLastError();
}

#define QMLP_MFGU(G_, MT_)                                                                \
    if (b.gg == G_ && MT == MT_) {                                                        \
        auto k = mf_gu_kernel<G_, MT_, kMfWaves>;                                         \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, kMfWaves * 64, lds, st>>>(b, nb);                                       \
        return hipGetLastError();                                                         \
    }

hipError_t launch_gateup_mfma(const BatchArgs& b, int nb, hipStream_t st) {
    if (!mfma_supported(b.M, b.d, b.f, b.gg, b.bg, b.gd, b.bd, b.r, nb))
        return hipErrorInvalidValue;
    const int MT = mf_mt(b.M);
    const int grid = mf_grid((long)nb * (b.f / 16));
    const size_t lds = mf_gu_lds(b.d, b.gg, MT);
    QMLP_MFGU(64, 4) QMLP_MFGU(64, 8) QMLP_MFGU(64, 16)
    QMLP_MFGU(128, 4) QMLP_MFGU(128, 8) QMLP_MFGU(128, 16)
    return hipErrorInvalidValue;
}

#define QMLP_MFDN(G_, MT_)                                                                \
    if (b.gd == G_ && MT == MT_) {                                                        \
        auto k = mf_dn_kernel<G_, MT_, dn_tpw(MT_), dn_waves(MT_), mf_stage_words(G_)>;   \
        hipError_t e = set_lds(k, lds);                                                   \
        if (e != hipSuccess) return e;                                                    \
        k<<<grid, dn_waves(MT_) * 64, lds, st>>>(b, nb, ck);                              \
        return hipGetLastError();                                                         \
    }

hipError_t launch_down_mfma(const BatchArgs& b, int nb, hipStream_t st) {
    if (!mfma_supported(b.M, b.d, b.f, b.gg, b.bg, b.gd, b.bd, b.r, nb))
        return hipErrorInvalidValue;
    const int MT = mf_mt(b.M);
    const int grid = mf_grid((long)nb * (b.d / 16));
    const int ck = mf_dn_chunk(b.f, b.gd, MT);
    const size_t lds = mf_dn_lds(ck, b.gd, MT);
    QMLP_MFDN(64, 4) QMLP_MFDN(64, 8) QMLP_MFDN(64, 16)
    QMLP_MFDN(128, 4) QMLP_MFDN(128, 8) QMLP_MFDN(128, 16)
    return hipErrorInvalidValue;
}

}  // namespace qmlp

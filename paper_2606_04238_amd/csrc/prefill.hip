// Prefill-chunk path of libqmlp (gfx950): M a multiple of 128 tokens,
// bfloat16 activations.  At this size the block is a dense contraction
// (Sec. 3.3 gated MLP over the quantized weights, Sec. 3.1 Eq. (1) for the
// adapters), so it runs on the matrix cores: weight tiles are dequantized to
// bfloat16 in LDS and multiplied with v_mfma_f32_32x32x16_bf16 (fp32
// accumulation).
//
// Kernels (stream order):
//   pf_lora_a  : partial t over a slice of the input dimension (split K),
//   pf_lora_t  : t = lora_scale * sum of the partials, rounded to bfloat16,
//   pf_gateup  : G, U tiles + the rank-r LoRA products + SiLU(G) * U -> h,
//   pf_down    : y = dequant4(W_down) h, split over S slices of f when the
//                token x row tiles alone would not fill the chip (fp32
//                partials [S][M][d]),
//   pf_down_reduce (S > 1): y = the partials' sum in slice order.
//
// Tile engine shared by the three GEMM kernels: a block of NT threads owns
// a BM-token x BN-weight-row tile (BM = 128 on 4 waves, or 256 on 8 waves
// where M allows) and walks the input dimension in steps of 64.  Each step
// stages the activation tile (BM x 64 bf16) and the dequantized weight tile
// (BN x 64 bf16) in LDS, rows of eight 16-byte chunks with chunk c of row r
// stored at c ^ ((r >> 1) & 7): the 16-byte fragment reads of an MFMA (32
// rows, one chunk) and the row-wise tile writes cover every LDS bank once
// per 16 lanes (two rows share a 256-byte bank line).  Two LDS buffers and
// one set of staging registers: while step k runs on the matrix cores the
// registers hold step k + 1, which then goes to the other buffer, and the
// global loads of step k + 2 are issued (one barrier per step).
#include "qmlp_device.h"
#include "qmlp_internal.h"
#include "decode_launch.h"

namespace qmlp {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int PF_BM = 128;     // tokens per block tile
constexpr int PF_BK = 64;      // input elements per step
constexpr int PF_NT = 256;     // threads per block

__device__ __forceinline__ int swz(int r, int c) { return r * 8 + (c ^ ((r >> 1) & 7)); }

// 16-byte global load / LDS store through a plain vector type (HIP's uint4
// copies are lowered to memcpy, which keeps a register tile in scratch).
__device__ __forceinline__ uint4 ld16(const void* p) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(p);
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st16(uint4* p, const uint4& v) {
    *reinterpret_cast<u32x4*>(p) = u32x4{v.x, v.y, v.z, v.w};
}

// Two fp32 values rounded to bfloat16 (nearest-even), packed low/high.
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ f32x16_t mfma(const uint4& a, const uint4& b, const f32x16_t& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// ------------------------------------------------------------ activation tile
// BM rows x 64 bf16 = 8 BM chunks, 4 per thread (BM = NT / 2); chunk id =
// tid + NT i.
struct ActRegs {
    uint4 v[4];
};

template <int NT = PF_NT>
__device__ __forceinline__ void act_load(ActRegs& ar, const uint16_t* A, int K, int m0, int k0,
                                         int tid) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int id = tid + NT * i, row = id >> 3, c = id & 7;
        ar.v[i] = ld16(A + (long)(m0 + row) * K + k0 + c * 8);
    }
}

template <int NT = PF_NT>
__device__ __forceinline__ void act_store(uint4* lds, const ActRegs& ar, int tid) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int id = tid + NT * i;
        st16(&lds[swz(id >> 3, id & 7)], ar.v[i]);
    }
}

// --------------------------------------------------------- quantized weights
// Thread t owns tile row t / P and part t % P (CPT = 64 / P codes) of a
// 128-row tile: P = 2 at 256 threads, 4 at 512.
template <int BITS, int CPT>
struct QRegs {
    uint32_t w[BITS * CPT / 32];   // CPT codes
    uint32_t meta;                 // scale | zero << 16 of the row's group
};

template <int BITS, int CPT>
__device__ __forceinline__ void q_load(QRegs<BITS, CPT>& qr, const uint32_t* codes_row,
                                       const uint32_t* meta_row, int k0, int g, int part) {
    constexpr int NW = BITS * CPT / 32;
    const uint32_t* p = codes_row + (k0 + part * CPT) * BITS / 32;
    if constexpr (NW == 1) {
        qr.w[0] = *p;
    } else if constexpr (NW == 2) {
        const uint2 v = *reinterpret_cast<const uint2*>(p);
        qr.w[0] = v.x;
        qr.w[1] = v.y;
    } else {
        const uint4 v = ld16(p);
        qr.w[0] = v.x;
        qr.w[1] = v.y;
        qr.w[2] = v.z;
        qr.w[3] = v.w;
    }
    qr.meta = meta_row[k0 / g];
}

// Dequantize CPT codes to bfloat16 scale * (q - zero) (one rounding: the fp32
// value is exact, since scale has 11 significant bits and |q - zero| < 16)
// and store them as chunks part * CPT/8 .. of the tile row.
template <int BITS, int CPT>
__device__ __forceinline__ void q_store(uint4* lds, const QRegs<BITS, CPT>& qr, int row, int part) {
    const float s = h2f(qr.meta & 0xFFFFu);
    const float nsz = -s * h2f(qr.meta >> 16);
    constexpr int C0 = CPT / 8;                     // chunks per thread
    if constexpr (BITS == 2) {
#pragma unroll
        for (int wi = 0; wi < CPT / 16; ++wi) {
            // byte b of m[i] holds code 4b + i of the word
            uint32_t m[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) m[i] = (qr.w[wi] >> (2 * i)) & 0x03030303u;
            float v[16];
#pragma unroll
            for (int c = 0; c < 16; ++c)
                v[c] = __builtin_fmaf((float)((m[c & 3] >> (8 * (c >> 2))) & 0xFFu), s, nsz);
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const uint4 o = make_uint4(pack_bf16(v[8 * j + 0], v[8 * j + 1]),
                                           pack_bf16(v[8 * j + 2], v[8 * j + 3]),
                                           pack_bf16(v[8 * j + 4], v[8 * j + 5]),
                                           pack_bf16(v[8 * j + 6], v[8 * j + 7]));
                st16(&lds[swz(row, part * C0 + wi * 2 + j)], o);
            }
        }
    } else {
#pragma unroll
        for (int wi = 0; wi < CPT / 8; ++wi) {
            // byte b of m0 holds code 2b, of m1 code 2b + 1
            const uint32_t m0 = qr.w[wi] & 0x0F0F0F0Fu, m1 = (qr.w[wi] >> 4) & 0x0F0F0F0Fu;
            float v[8];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                v[2 * b] = __builtin_fmaf((float)((m0 >> (8 * b)) & 0xFFu), s, nsz);
                v[2 * b + 1] = __builtin_fmaf((float)((m1 >> (8 * b)) & 0xFFu), s, nsz);
            }
            st16(&lds[swz(row, part * C0 + wi)],
                 make_uint4(pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3]), pack_bf16(v[4], v[5]),
                            pack_bf16(v[6], v[7])));
        }
    }
}

// ------------------------------------------------------------- MFMA step
// One 64-wide step over LDS tiles: wave (wm, wn) multiplies its WM 32-row
// activation tiles with its WN 32-row weight tiles.
template <int WM, int WN>
__device__ __forceinline__ void mfma_step(const uint4* xs, const uint4* ws, f32x16_t (&acc)[WM][WN],
                                          int wm, int wn, int lane) {
    const int r = lane & 31, hk = lane >> 5;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        uint4 a[WM], b[WN];
#pragma unroll
        for (int i = 0; i < WM; ++i) a[i] = ld16(&xs[swz(wm * 32 * WM + i * 32 + r, 2 * s + hk)]);
#pragma unroll
        for (int j = 0; j < WN; ++j) b[j] = ld16(&ws[swz(wn * 32 * WN + j * 32 + r, 2 * s + hk)]);
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int j = 0; j < WN; ++j) acc[i][j] = mfma(a[i], b[j], acc[i][j]);
    }
}

// Row of accumulator element v of lane `lane` within a 32 x 32 tile (the
// column is lane & 31).
__device__ __forceinline__ int acc_row(int v, int lane) {
    return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
}

// ------------------------------------------------------------ kernels
struct PfGateUpArgs {
    const uint32_t *cg, *mg, *cu, *mu;   // gate / up codes and meta
    const uint16_t* x;                    // [M][d] bf16
    const uint16_t* T;                    // [M][2r] bf16: lora_scale * (A_g x, A_u x)
    const uint16_t *Bg, *Bu;              // [f][r] bf16
    uint16_t* h;                          // [M][f] bf16
    int M, d, f, g, r;
};

// Block tile: BM tokens x HC columns of h.  The 2 HC weight rows come in
// groups of 64: gate rows c..c+31 then up rows c..c+31 of the group's 32
// columns c, so a wave tile of 32 WM tokens x one group holds G and U of the
// same outputs.  Waves: BM / (32 WM) along tokens x HC / 32 along columns.
template <int BM, int HC, int NT, int WM>
__global__ void __launch_bounds__(NT) pf_gateup_kernel(PfGateUpArgs a) {
    constexpr int BN = 2 * HC, WMW = BM / (32 * WM), P = NT / BN, CPT = 64 / P;
    static_assert(NT == 2 * BM, "4 activation chunks per thread");
    static_assert(WMW * (HC / 32) == NT / 64, "one wave tile per wave");
    extern __shared__ uint4 smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WMW, wn = wave / WMW;
    const int mtiles = a.M / BM;
    const int mt0 = blockIdx.x % mtiles, nt0 = blockIdx.x / mtiles;
    const int m0 = mt0 * BM, n0 = nt0 * HC;

    const int trow = tid / P, part = tid % P;
    const int mat = (trow >> 5) & 1;
    const int wrow = n0 + (trow >> 6) * 32 + (trow & 31);
    const int wpr = a.d / 16, ng = a.d / a.g;
    const uint32_t* crow = (mat ? a.cu : a.cg) + (long)wrow * wpr;
    const uint32_t* mrow = (mat ? a.mu : a.mg) + (long)wrow * ng;

    f32x16_t acc[WM][2];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

    // Step k's tiles are staged during step k - 1's matrix-core work: the
    // MFMAs of a step are issued, then the same wave dequantizes and stores
    // the next step's tiles into the other buffer while they run.  One
    // barrier per step: step k's tiles are complete, and every wave is done
    // reading the buffer step k + 1 will overwrite.
    ActRegs ar;
    QRegs<2, CPT> qr;
    const int nk = a.d / PF_BK;
    act_load<NT>(ar, a.x, a.d, m0, 0, tid);
    q_load<2, CPT>(qr, crow, mrow, 0, a.g, part);
    act_store<NT>(smem, ar, tid);
    q_store<2, CPT>(smem + BM * 8, qr, trow, part);
    {
        const int k1 = (nk > 1 ? 1 : 0) * PF_BK;
        act_load<NT>(ar, a.x, a.d, m0, k1, tid);
        q_load<2, CPT>(qr, crow, mrow, k1, a.g, part);
    }
    for (int kt = 0; kt < nk; ++kt) {
        __syncthreads();
        uint4* xs = smem + (kt & 1) * (BM + BN) * 8;
        mfma_step<WM, 2>(xs, xs + BM * 8, acc, wm, wn, lane);
        // the next step's tiles (past the last step: a copy of the last
        // step's, never read), then the loads of the one after
        uint4* xn = smem + ((kt + 1) & 1) * (BM + BN) * 8;
        act_store<NT>(xn, ar, tid);
        q_store<2, CPT>(xn + BM * 8, qr, trow, part);
        const int k2 = (kt + 2 < nk ? kt + 2 : nk - 1) * PF_BK;
        act_load<NT>(ar, a.x, a.d, m0, k2, tid);
        q_load<2, CPT>(qr, crow, mrow, k2, a.g, part);
    }

    // LoRA: G += T_g B_g^T, U += T_u B_u^T over k < r (zero-padded to 16).
    if (a.r > 0) {
        const int r = lane & 31, hk = lane >> 5;
        const int ncol = n0 + wn * 32 + r;
        for (int s = 0; s * 16 < a.r; ++s) {
            const int kk = 16 * s + 8 * hk;
            const bool in = kk < a.r;
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const uint16_t* Bm = j ? a.Bu : a.Bg;
                const uint4 b = in ? ld16(Bm + (long)ncol * a.r + kk) : make_uint4(0, 0, 0, 0);
#pragma unroll
                for (int i = 0; i < WM; ++i) {
                    const int m = m0 + wm * 32 * WM + i * 32 + r;
                    const uint4 t = in ? ld16(a.T + (long)m * 2 * a.r + j * a.r + kk)
                                       : make_uint4(0, 0, 0, 0);
                    acc[i][j] = mfma(t, b, acc[i][j]);
                }
            }
        }
    }

    // SiLU(G) * U -> h (bf16)
    const int col = n0 + wn * 32 + (lane & 31);
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int m = m0 + wm * 32 * WM + i * 32 + acc_row(v, lane);
            const float G = acc[i][0][v], U = acc[i][1][v];
            const float hv = G / (1.0f + __expf(-G)) * U;
            const bf16x2_t p = {(__bf16)hv, (__bf16)0.0f};
            a.h[(long)m * a.f + col] = (uint16_t)(__builtin_bit_cast(uint32_t, p) & 0xFFFFu);
        }
}

struct PfDownArgs {
    const uint32_t *cd, *md;     // down codes [d][f/8], meta [d][f/g]
    const uint16_t* h;           // [M][f] bf16
    uint16_t* y;                 // [M][d] bf16 (S == 1)
    float* part;                 // [S][M][d] fp32 partial sums (S > 1)
    int M, d, f, g, S;           // S: slices of f (split K), f / S a multiple of 64
};

template <int BM, int NT>
__global__ void __launch_bounds__(NT) pf_down_kernel(PfDownArgs a) {
    constexpr int BN = 128, WMW = BM / 64, P = NT / 128, CPT = 64 / P;
    static_assert(NT == 2 * BM, "4 activation chunks per thread");
    extern __shared__ uint4 smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % WMW, wn = wave / WMW;
    const int mtiles = a.M / BM, ntiles = a.d / BN;
    const int sl = blockIdx.x / (mtiles * ntiles), tile = blockIdx.x - sl * mtiles * ntiles;
    const int mt0 = tile % mtiles, nt0 = tile / mtiles;
    const int m0 = mt0 * BM, n0 = nt0 * BN;
    const int kper = a.f / a.S, kbeg = sl * kper;     // this block's slice of f

    const int trow = tid / P, part = tid % P;
    const int wpr = a.f / 8, ng = a.f / a.g;
    const uint32_t* crow = a.cd + (long)(n0 + trow) * wpr;
    const uint32_t* mrow = a.md + (long)(n0 + trow) * ng;

    f32x16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

    // staged one step ahead, as in the gate/up kernel
    ActRegs ar;
    QRegs<4, CPT> qr;
    const int nk = kper / PF_BK;
    act_load<NT>(ar, a.h, a.f, m0, kbeg, tid);
    q_load<4, CPT>(qr, crow, mrow, kbeg, a.g, part);
    act_store<NT>(smem, ar, tid);
    q_store<4, CPT>(smem + BM * 8, qr, trow, part);
    {
        const int k1 = kbeg + (nk > 1 ? 1 : 0) * PF_BK;
        act_load<NT>(ar, a.h, a.f, m0, k1, tid);
        q_load<4, CPT>(qr, crow, mrow, k1, a.g, part);
    }
    for (int kt = 0; kt < nk; ++kt) {
        __syncthreads();
        uint4* xs = smem + (kt & 1) * (BM + BN) * 8;
        mfma_step<2, 2>(xs, xs + BM * 8, acc, wm, wn, lane);
        uint4* xn = smem + ((kt + 1) & 1) * (BM + BN) * 8;
        act_store<NT>(xn, ar, tid);
        q_store<4, CPT>(xn + BM * 8, qr, trow, part);
        const int k2 = kbeg + (kt + 2 < nk ? kt + 2 : nk - 1) * PF_BK;
        act_load<NT>(ar, a.h, a.f, m0, k2, tid);
        q_load<4, CPT>(qr, crow, mrow, k2, a.g, part);
    }

    float* out = a.S > 1 ? a.part + (long)sl * a.M * a.d : nullptr;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int col = n0 + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * 64 + i * 32 + acc_row(v, lane);
                if (out) {
                    out[(long)m * a.d + col] = acc[i][j][v];
                } else {
                    const bf16x2_t p = {(__bf16)acc[i][j][v], (__bf16)0.0f};
                    a.y[(long)m * a.d + col] = (uint16_t)(__builtin_bit_cast(uint32_t, p) & 0xFFFFu);
                }
            }
    }
}

// y[i] = bf16(sum of the S <= kDownSlicesMax partials, in slice order), four
// outputs per thread with 16-byte loads (n % 4 == 0).
constexpr int kDownSlicesMax = 8;
__global__ void pf_down_reduce_kernel(const float* part, uint16_t* y, long n, int S) {
    const long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
    if (i >= n)
        return;
    float s0 = 0.0f, s1 = 0.0f, s2 = 0.0f, s3 = 0.0f;
    for (int k = 0; k < S; ++k) {
        const f32x4_t v = *reinterpret_cast<const f32x4_t*>(part + (long)k * n + i);
        s0 += v[0];
        s1 += v[1];
        s2 += v[2];
        s3 += v[3];
    }
    *reinterpret_cast<uint2*>(y + i) = make_uint2(pack_bf16(s0, s1), pack_bf16(s2, s3));
}

struct PfLoraArgs {
    const uint16_t *Ag, *Au;     // [r][d] bf16
    const uint16_t* x;           // [M][d] bf16
    float* part;                 // [S][M][2r] fp32
    int M, d, r, S;
};

// Partial t over one of S slices of the input dimension: a 128-token x
// 64-row tile (rows >= 2r are zero).
__global__ void __launch_bounds__(PF_NT) pf_lora_a_kernel(PfLoraArgs a) {
    constexpr int BN = 64;
    __shared__ uint4 lds[2][(PF_BM + BN) * 8];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1, wn = wave >> 1;
    const int mtiles = a.M / PF_BM;
    const int mt0 = blockIdx.x % mtiles, sl = blockIdx.x / mtiles;
    const int m0 = mt0 * PF_BM;
    const int nk = a.d / PF_BK / a.S, kbeg = sl * nk * PF_BK;

    f32x16_t acc[2][1];
    acc[0][0] = f32x16_t{};
    acc[1][0] = f32x16_t{};

    // weight rows: 64 rows x 8 chunks = 2 chunks per thread (rows >= 2r read
    // row 0 and are zeroed)
    const uint16_t* src[2];
    uint32_t live[2];                   // all ones for rows < 2r, else zero
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int id = tid + PF_NT * i, row = id >> 3, c = id & 7;
        live[i] = row < 2 * a.r ? ~0u : 0u;
        const uint16_t* base = row >= 2 * a.r ? a.Ag : row < a.r ? a.Ag + (long)row * a.d
                                                                  : a.Au + (long)(row - a.r) * a.d;
        src[i] = base + c * 8;
    }
    auto masked = [](uint4 v, uint32_t m) { return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m); };
    ActRegs ar;
    uint4 wv[2];
    act_load(ar, a.x, a.d, m0, kbeg, tid);
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        wv[i] = masked(ld16(src[i] + kbeg), live[i]);
    }
    for (int kt = 0; kt < nk; ++kt) {
        uint4* xs = lds[kt & 1];
        uint4* ws = xs + PF_BM * 8;
        act_store(xs, ar, tid);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int id = tid + PF_NT * i;
            st16(&ws[swz(id >> 3, id & 7)], wv[i]);
        }
        __syncthreads();
        {
            const int k1 = kbeg + (kt + 1 < nk ? kt + 1 : kt) * PF_BK;
            act_load(ar, a.x, a.d, m0, k1, tid);
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                wv[i] = masked(ld16(src[i] + k1), live[i]);
            }
        }
        mfma_step<2, 1>(xs, ws, acc, wm, wn, lane);
    }
    const int c = wn * 32 + (lane & 31);
    if (c < 2 * a.r) {
        float* out = a.part + (long)sl * a.M * 2 * a.r;
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + wm * 64 + i * 32 + acc_row(v, lane);
                out[(long)m * 2 * a.r + c] = acc[i][0][v];
            }
    }
}

// T[m][c] = bf16(lora_scale * sum over the S <= kLoraSplitsMax slices, in
// slice order).
constexpr int kLoraSplitsMax = 24;
__global__ void pf_lora_t_kernel(const float* part, uint16_t* T, int M, int r, int S,
                                 float lora_scale) {
    const long n = (long)M * 2 * r;
    const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n)
        return;
    // every load first (slots past S re-read slice S - 1 and are dropped),
    // then the sum in slice order
    float v[kLoraSplitsMax];
#pragma unroll
    for (int k = 0; k < kLoraSplitsMax; ++k) v[k] = part[(long)(k < S ? k : S - 1) * n + i];
    float s = 0.0f;
#pragma unroll
    for (int k = 0; k < kLoraSplitsMax; ++k)
        if (k < S)
            s += v[k];
    const bf16x2_t p = {(__bf16)(lora_scale * s), (__bf16)0.0f};
    T[i] = (uint16_t)(__builtin_bit_cast(uint32_t, p) & 0xFFFFu);
}

}  // namespace

bool prefill_supported(int M, int d, int f, int g, int r) {
    (void)g;
    (void)r;
    return M > 0 && M % PF_BM == 0 && d % 128 == 0 && f % 64 == 0;
}

int prefill_splits(int d) {
    const int nk = d / PF_BK;
    for (int s = nk < kLoraSplitsMax ? nk : kLoraSplitsMax; s > 1; --s)
        if (nk % s == 0 && nk / s >= 2)
            return s;
    return 1;
}

hipError_t launch_prefill_lora(const uint16_t* Ag, const uint16_t* Au, const uint16_t* x, int M,
                               int d, int r, float lora_scale, float* part, uint16_t* T,
                               hipStream_t st) {
    const int S = prefill_splits(d);
    PfLoraArgs a{Ag, Au, x, part, M, d, r, S};
    pf_lora_a_kernel<<<(M / PF_BM) * S, PF_NT, 0, st>>>(a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const long n = (long)M * 2 * r;
    pf_lora_t_kernel<<<(unsigned)((n + 255) / 256), 256, 0, st>>>(part, T, M, r, S, lora_scale);
    return hipGetLastError();
}

// Token tile of the gate/up and down kernels: 256 tokens (8 waves; every
// dequantized weight serves 256 tokens) where M allows, else 128 (4 waves).
int prefill_bm(int M) { return M % 256 == 0 ? 256 : 128; }
hipError_t launch_prefill_gateup(const uint32_t* cg, const uint32_t* mg, const uint32_t* cu,
                                 const uint32_t* mu, const uint16_t* x, const uint16_t* T,
                                 const uint16_t* Bg, const uint16_t* Bu, uint16_t* h, int M, int d,
                                 int f, int g, int r, hipStream_t st) {
    PfGateUpArgs a{cg, mg, cu, mu, x, T, Bg, Bu, h, M, d, f, g, r};
    const int BM = prefill_bm(M);
    // 256 tokens x 128 columns of h (wave tiles of 128 tokens x 32 columns,
    // half the LDS reads and two thirds of the LDS writes per MFMA of the
    // 64-column tile) where f allows
    const int HC = BM == 256 && f % 128 == 0 ? 128 : 64;
    const size_t lds = (size_t)2 * (BM + 2 * HC) * 8 * 16;
    auto run = [&](auto k) {
        hipError_t e = set_lds(k, lds);
        if (e != hipSuccess)
            return e;
        k<<<(M / BM) * (f / HC), 2 * BM, lds, st>>>(a);
        return hipGetLastError();
    };
    if (HC == 128)
        return run(pf_gateup_kernel<256, 128, 512, 4>);
    return BM == 256 ? run(pf_gateup_kernel<256, 64, 512, 2>) : run(pf_gateup_kernel<128, 64, 256, 2>);
}

int prefill_down_slices(int M, int d, int f) {
    // Enough (token tile x row tile x slice) blocks for two rounds over the
    // compute units; slices of f stay whole 64-wide steps.
    const long tiles = (long)(M / prefill_bm(M)) * (d / 128);
    int S = 1;
    while (S < kDownSlicesMax && tiles * S < 512 && f % (2 * S * PF_BK) == 0) S *= 2;
    return S;
}

size_t prefill_down_part_bytes(int M, int d, int f) {
    const int S = prefill_down_slices(M, d, f);
    return S > 1 ? (size_t)S * M * d * 4 : 0;
}

hipError_t launch_prefill_down(const uint32_t* cd, const uint32_t* md, const uint16_t* h,
                               uint16_t* y, int M, int d, int f, int g, float* part, hipStream_t st) {
    const int S = part ? prefill_down_slices(M, d, f) : 1;
    PfDownArgs a{cd, md, h, y, part, M, d, f, g, S};
    const int BM = prefill_bm(M);
    const size_t lds = (size_t)2 * (BM + 128) * 8 * 16;
    auto run = [&](auto k) {
        hipError_t e = set_lds(k, lds);
        if (e != hipSuccess)
            return e;
        k<<<(M / BM) * (d / 128) * S, 2 * BM, lds, st>>>(a);
        return hipGetLastError();
    };
    hipError_t e = BM == 256 ? run(pf_down_kernel<256, 512>) : run(pf_down_kernel<128, 256>);
    if (e != hipSuccess || S == 1)
        return e;
    const long n = (long)M * d;                          // d % 128 == 0
    pf_down_reduce_kernel<<<(unsigned)((n / 4 + 255) / 256), 256, 0, st>>>(part, y, n, S);
    return hipGetLastError();
}

}  // namespace qmlp

// Offline packing, unpacking and dequantization kernels (gfx950).
//
// Quantizer: the paper fixes bits and group size only (Sec. 3.3: gate/up
// INT2, every other linear INT4, group-wise; Sec. 4.1: Stage 1 post-training
// quantization).  This library reads it as round-to-nearest asymmetric
// min-max with an integer zero point and a binary16 scale; the arithmetic is
// IEEE fp64 with exactly one rounding of the scale to binary16, so every
// code, scale and zero is reproducible bit for bit.
#include "qmlp_device.h"
#include "qmlp_internal.h"

#pragma clang fp contract(off)

namespace qmlp {

// fp64 -> binary16 bits, a single round-to-nearest-even (never through fp32).
// Built from the bit fields of the double.
__device__ uint32_t f64_to_f16_bits(double v) {
    const uint64_t b = __builtin_bit_cast(uint64_t, v);
    const uint32_t sign = (uint32_t)(b >> 48) & 0x8000u;
    const int e = (int)((b >> 52) & 0x7FF);
    const uint64_t frac = b & ((1ull << 52) - 1);
    if (e == 0x7FF)
        return frac ? 0x7E00u : (sign | 0x7C00u);
    if (e == 0)
        return sign;                       // fp64 subnormal: far below 2^-25
    const int E = e - 1023;                // value = 1.frac * 2^E
    if (E > 15)
        return sign | 0x7C00u;
    uint64_t keep, rest, halfway;
    int shift;
    uint64_t mant = (1ull << 52) | frac;   // 53-bit significand
    if (E >= -14) {
        shift = 42;                        // keep 11 bits (implicit one + 10)
    } else {
        shift = 42 + (-14 - E);            // subnormal: quantum 2^-24
        if (shift > 63)
            return sign;                   // below half the smallest subnormal
    }
    keep = mant >> shift;
    rest = mant & ((1ull << shift) - 1);
    halfway = 1ull << (shift - 1);
    if (rest > halfway || (rest == halfway && (keep & 1)))
        ++keep;
    if (E >= -14) {
        int he = E + 15;
        if (keep == 2048) {                // rounded up to the next binade
            keep = 1024;
            ++he;
        }
        if (he >= 31)
            return sign | 0x7C00u;
        return sign | ((uint32_t)he << 10) | (uint32_t)(keep - 1024);
    }
    return sign | (uint32_t)keep;          // keep == 1024 is 2^-14, still correct
}

__device__ double f16_bits_to_f64(uint32_t h) { return (double)h2f(h); }

// One thread per (row, group).  W is [n][k] fp32; codes row-major words;
// meta one uint32 per group: scale bits low, zero bits high.
// 3 bits (Appendix B): a row is two planes, the low two bits of every code
// in the 2-bit layout (k/16 words) followed by the high bit of every code
// (k/32 words, code i at bit i mod 32 of word i/32 of the plane).
template <int BITS>
__global__ void __launch_bounds__(256)
pack_kernel(const float* __restrict__ W, int n, int k, int g,
            uint32_t* __restrict__ codes, uint32_t* __restrict__ meta, int32_t* status) {
    constexpr int QMAX = (1 << BITS) - 1;
    constexpr int PER = BITS == 3 ? 16 : 32 / BITS;       // codes per word (of the 2-bit plane)
    const int ng = k / g;
    const long gid = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= (long)n * ng)
        return;
    const long row = gid / ng;
    const long j = gid - row * ng;
    const float* w = W + row * (long)k + j * (long)g;
    const long row_words = BITS == 3 ? (long)k * 3 / 32 : (long)(k / PER);
    uint32_t* out = codes + row * row_words + j * (long)(g / PER);
    uint32_t* out_hi = codes + row * row_words + k / 16 + j * (long)(g / 32);   // 3 bits only

    bool finite = true;
    double lo = 0.0, hi = 0.0;
    for (int i = 0; i < g; ++i) {
        const double v = (double)w[i];
        if (!__builtin_isfinite(v)) {
            finite = false;
        } else {
            if (v < lo) lo = v;
            if (v > hi) hi = v;
        }
    }
    const double s = (hi - lo) / (double)QMAX;
    uint32_t s16 = f64_to_f16_bits(s);
    if (s16 == 0)
        s16 = 0x3C00u;                     // degenerate range: scale 1.0
    if (!finite || s16 == 0x7C00u) {
        for (int wd = 0; wd < g / PER; ++wd)
            out[wd] = 0;
        if (BITS == 3)
            for (int wd = 0; wd < g / 32; ++wd)
                out_hi[wd] = 0;
        meta[gid] = 0x00007E00u;           // scale NaN, zero 0
        if (status)
            atomicOr(status, 1);
        return;
    }
    const double sd = f16_bits_to_f64(s16);
    double zf = __builtin_rint(-lo / sd);
    zf = zf < 0.0 ? 0.0 : (zf > (double)QMAX ? (double)QMAX : zf);
    const int z = (int)zf;
    uint32_t hbits = 0;                       // 3 bits: high bits of the current 32 codes
    for (int wd = 0; wd < g / PER; ++wd) {
        uint32_t word = 0;
        for (int i = 0; i < PER; ++i) {
            double t = __builtin_rint((double)w[wd * PER + i] / sd) + (double)z;
            t = t < 0.0 ? 0.0 : (t > (double)QMAX ? (double)QMAX : t);
            const uint32_t q = (uint32_t)t;
            if (BITS == 3) {
                word |= (q & 3u) << (2 * i);
                hbits |= (q >> 2) << ((wd * PER + i) & 31);
                if (((wd * PER + i) & 31) == 31) {
                    out_hi[(wd * PER + i) >> 5] = hbits;
                    hbits = 0;
                }
            } else {
                word |= q << (BITS * i);
            }
        }
        out[wd] = word;
    }
    meta[gid] = s16 | (f2h((float)z) << 16);
}

// One thread per 32-bit code word: canonical codes uint8 [n][k]; the thread
// holding the first word of a group also writes that group's scale and zero.
// Code i of a word: BITS-bit field i; at 3 bits the 2-bit field of the low
// plane and the bit of the high plane (code_word: the low-plane word, hi:
// the high-plane bits of the same 16 codes, in bits 0-15).
template <int BITS>
__device__ __forceinline__ uint32_t code_at(uint32_t code_word, uint32_t hi, int i) {
    if (BITS == 3)
        return ((code_word >> (2 * i)) & 3u) | (((hi >> i) & 1u) << 2);
    return (code_word >> (BITS * i)) & ((1u << BITS) - 1);
}

// The word of the (low) plane at word index gid of the row-major view, the
// row and first code column it covers, and the matching high-plane bits.
template <int BITS>
__device__ __forceinline__ void word_at(const uint32_t* codes, int k, long gid, uint32_t& wv,
                                        uint32_t& hi, long& row, long& col) {
    constexpr int PER = BITS == 3 ? 16 : 32 / BITS;
    row = gid / (k / PER);
    col = (gid - row * (k / PER)) * PER;
    const long row_words = BITS == 3 ? (long)k * 3 / 32 : (long)(k / PER);
    wv = codes[row * row_words + col / PER];
    hi = BITS == 3 ? codes[row * row_words + k / 16 + col / 32] >> (col & 31) : 0u;
}

template <int BITS>
__global__ void __launch_bounds__(256)
unpack_kernel(const uint32_t* __restrict__ codes, const uint32_t* __restrict__ meta,
              int n, int k, int g, uint8_t* __restrict__ out_codes,
              uint16_t* __restrict__ scales, uint16_t* __restrict__ zeros) {
    constexpr int PER = BITS == 3 ? 16 : 32 / BITS;
    const long words = (long)n * (k / PER);
    const long gid = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= words)
        return;
    uint32_t w, hi;
    long row, col;                                    // col: first code index in the row
    word_at<BITS>(codes, k, gid, w, hi, row, col);
    uint8_t* dst = out_codes + row * (long)k + col;
    for (int i = 0; i < PER; ++i)
        dst[i] = (uint8_t)code_at<BITS>(w, hi, i);
    if (col % g == 0) {
        const long gi = row * (k / g) + col / g;
        const uint32_t m = meta[gi];
        scales[gi] = (uint16_t)(m & 0xFFFFu);
        zeros[gi] = (uint16_t)(m >> 16);
    }
}

// One thread per code word: w_hat = scale * (q - zero) is exact in fp32
// (an 11-bit scale times an integer below 16), then one nearest-even
// rounding to binary16.  A NaN scale (invalid group) yields 0x7E00.
template <int BITS>
__global__ void __launch_bounds__(256)
dequant_kernel(const uint32_t* __restrict__ codes, const uint32_t* __restrict__ meta,
               int n, int k, int g, uint16_t* __restrict__ out) {
    constexpr int PER = BITS == 3 ? 16 : 32 / BITS;
    const long words = (long)n * (k / PER);
    const long gid = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (gid >= words)
        return;
    uint32_t w, hi;
    long row, col;
    word_at<BITS>(codes, k, gid, w, hi, row, col);
    const uint32_t m = meta[row * (k / g) + col / g];
    const float s = h2f(m & 0xFFFFu);
    const float z = h2f(m >> 16);
    const bool nan_scale = (m & 0x7C00u) == 0x7C00u && (m & 0x03FFu) != 0;
    uint16_t* dst = out + row * (long)k + col;
    for (int i = 0; i < PER; ++i) {
        const float q = (float)code_at<BITS>(w, hi, i);
        const float v = s * (q - z) + 0.0f;
        dst[i] = nan_scale ? (uint16_t)0x7E00u : (uint16_t)f2h(v);
    }
}

static inline unsigned blocks_for(long threads) { return (unsigned)((threads + 255) / 256); }

hipError_t launch_pack(int bits, const float* W, int n, int k, int g, uint32_t* codes,
                       uint32_t* meta, int32_t* status, hipStream_t st) {
    const long groups = (long)n * (k / g);
    if (bits == 2)
        pack_kernel<2><<<blocks_for(groups), 256, 0, st>>>(W, n, k, g, codes, meta, status);
    else if (bits == 3)
        pack_kernel<3><<<blocks_for(groups), 256, 0, st>>>(W, n, k, g, codes, meta, status);
    else
        pack_kernel<4><<<blocks_for(groups), 256, 0, st>>>(W, n, k, g, codes, meta, status);
    return hipGetLastError();
}

hipError_t launch_unpack(int bits, const uint32_t* codes, const uint32_t* meta, int n, int k,
                         int g, uint8_t* out_codes, uint16_t* scales, uint16_t* zeros,
                         hipStream_t st) {
    const long words = (long)n * (k / (bits == 4 ? 8 : 16));
    if (bits == 2)
        unpack_kernel<2><<<blocks_for(words), 256, 0, st>>>(codes, meta, n, k, g, out_codes,
                                                             scales, zeros);
    else if (bits == 3)
        unpack_kernel<3><<<blocks_for(words), 256, 0, st>>>(codes, meta, n, k, g, out_codes,
                                                             scales, zeros);
    else
        unpack_kernel<4><<<blocks_for(words), 256, 0, st>>>(codes, meta, n, k, g, out_codes,
                                                             scales, zeros);
    return hipGetLastError();
}

hipError_t launch_dequant(int bits, const uint32_t* codes, const uint32_t* meta, int n, int k,
                          int g, uint16_t* out, hipStream_t st) {
    const long words = (long)n * (k / (bits == 4 ? 8 : 16));
    if (bits == 2)
        dequant_kernel<2><<<blocks_for(words), 256, 0, st>>>(codes, meta, n, k, g, out);
    else if (bits == 3)
        dequant_kernel<3><<<blocks_for(words), 256, 0, st>>>(codes, meta, n, k, g, out);
    else
        dequant_kernel<4><<<blocks_for(words), 256, 0, st>>>(codes, meta, n, k, g, out);
    return hipGetLastError();
}

}  // namespace qmlp

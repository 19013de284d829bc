// Device-side helpers shared by the gfx950 kernels of libqmlp.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace qmlp {

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// 128-bit streaming load of weights that are read once per call (non-temporal
// hint: do not keep the lines in the caches).
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint32_t load_stream(const uint32_t* p) {
    return __builtin_nontemporal_load(p);
}

// Exact binary16 bits -> fp32.
__device__ __forceinline__ float h2f(uint32_t bits16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
}

// fp32 -> binary16 bits, round to nearest even (v_cvt_f16_f32 in the default mode).
__device__ __forceinline__ uint32_t f2h(float v) {
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v);
}

// Two fp16 lanes of a, b multiplied pairwise and added to c in fp32
// (v_dot2_f32_f16).
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2(__builtin_bit_cast(half2_t, a), __builtin_bit_cast(half2_t, b),
                                  c, false);
}

// Integer codes placed into the fraction of binary16 1024.0 (0x6400): a half
// holding code q at fraction bits [j, j+b) reads 1024 + q * 2^j exactly.
// One v_and_or_b32 yields two codes (one per half).  Codes are moved to the
// top of the fraction (j >= 4) so the 1024 offset, removed after the fp32
// dot products, stays small next to the code term (the cancellation error
// of the fp32 accumulation shrinks with 2^j).
__device__ __forceinline__ uint32_t magic(uint32_t w, uint32_t mask) {
    return (w & mask) | 0x64006400u;
}

// Code pairs of one 32-bit word of 2-bit codes (code i at bits 2i).  Pair p
// holds (code p, code 8+p) at fraction bits 2k(p), k(p) = {2,3,2,3,4,2,3,4},
// i.e. each half reads 1024 + q * 4^k(p).  Two shifts + eight and-or.
__device__ __forceinline__ void extract_w2(uint32_t w, uint32_t e[8]) {
    const uint32_t l = w << 4;          // codes 0,1 -> bits 4-7
    const uint32_t r = w >> 6;          // codes 5,6,7 -> bits 4-9
    e[0] = magic(l, 0x00300030u);
    e[1] = magic(l, 0x00C000C0u);
    e[2] = magic(w, 0x00300030u);
    e[3] = magic(w, 0x00C000C0u);
    e[4] = magic(w, 0x03000300u);
    e[5] = magic(r, 0x00300030u);
    e[6] = magic(r, 0x00C000C0u);
    e[7] = magic(r, 0x03000300u);
}

// 4^-k(p) for the 2-bit pair positions above (k packed 4 bits per pair).
__device__ __forceinline__ float w2_pair_scale(int p) {
    const int k = (0x43243232 >> (4 * p)) & 15;
    return __builtin_bit_cast(float, (uint32_t)(127 - 2 * k) << 23);
}

// Code pairs of one word of 4-bit codes (code i at bits 4i).  Pair p holds
// (code p, code 4+p): pairs 0,1 at fraction bits 4-7 (1024 + 16q), pairs 2,3
// at bits 6-9 (1024 + 64q).  Three shifts + four and-or.
__device__ __forceinline__ void extract_w4(uint32_t w, uint32_t e[4]) {
    e[0] = magic(w << 4, 0x00F000F0u);
    e[1] = magic(w, 0x00F000F0u);
    e[2] = magic(w >> 2, 0x03C003C0u);
    e[3] = magic(w >> 6, 0x03C003C0u);
}

// 16^-1 / 64^-1 for the 4-bit pair positions above.
__device__ __forceinline__ float w4_pair_scale(int p) { return p < 2 ? 1.0f / 16 : 1.0f / 64; }

// Opaque identity: the value is treated as redefined here, so work derived
// from registers preloaded before a loop is not hoisted out of the loop
// (which would keep every unpacked code live at once).
__device__ __forceinline__ void pin(uint32_t& v) { __asm__ volatile("" : "+v"(v)); }

// Sum over the `width` consecutive lanes sharing an output row (xor butterfly;
// every lane of the group ends with the total).
template <int WIDTH>
__device__ __forceinline__ float group_sum(float v) {
#pragma unroll
    for (int off = WIDTH / 2; off >= 1; off >>= 1)
        v += __shfl_xor(v, off, 64);
    return v;
}

}  // namespace qmlp

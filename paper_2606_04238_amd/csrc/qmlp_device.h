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
// With mv = magic_vgpr() (0x64006400 in a VGPR the compiler cannot see
// through) this is one v_and_or_b32, the mask in an SGPR: a VOP3 instruction
// on gfx950 reads at most one SGPR or literal, so with the constant as a
// literal the compiler splits the expression into v_and + v_or.
__device__ __forceinline__ uint32_t magic_vgpr() {
    uint32_t v;
    __asm__ volatile("v_mov_b32 %0, 0x64006400" : "=v"(v));
    return v;
}
__device__ __forceinline__ uint32_t magic(uint32_t w, uint32_t mask, uint32_t mv) {
    return (w & mask) | mv;
}

// Code pairs of one 32-bit word of 2-bit codes (code i at bits 2i).  Pair p
// holds (code p, code 8+p) at fraction bits 2k(p), k(p) = {2,3,2,3,4,2,3,4},
// i.e. each half reads 1024 + q * 4^k(p).  Two shifts + eight and-or.
__device__ __forceinline__ void extract_w2(uint32_t w, uint32_t e[8], uint32_t mv) {
    const uint32_t l = w << 4;          // codes 0,1 -> bits 4-7
    const uint32_t r = w >> 6;          // codes 5,6,7 -> bits 4-9
    e[0] = magic(l, 0x00300030u, mv);
    e[1] = magic(l, 0x00C000C0u, mv);
    e[2] = magic(w, 0x00300030u, mv);
    e[3] = magic(w, 0x00C000C0u, mv);
    e[4] = magic(w, 0x03000300u, mv);
    e[5] = magic(r, 0x00300030u, mv);
    e[6] = magic(r, 0x00C000C0u, mv);
    e[7] = magic(r, 0x03000300u, mv);
}

// The pair (bit i, bit 16 + i) of a word of 1-bit codes, moved to fraction
// bit 8 of the two halves: each reads 1024 + 256 b.
__device__ __forceinline__ uint32_t bit_pair(uint32_t w, int i, uint32_t mv) {
    const uint32_t v = i <= 8 ? w << (8 - i) : w >> (i - 8);
    return (v & 0x01000100u) | mv;
}

// 4^-k(p) for the 2-bit pair positions above (k packed 4 bits per pair).
__device__ __forceinline__ float w2_pair_scale(int p) {
    const int k = (0x43243232 >> (4 * p)) & 15;
    return __builtin_bit_cast(float, (uint32_t)(127 - 2 * k) << 23);
}

// Code pairs of one word of 4-bit codes (code i at bits 4i).  Pair p holds
// (code p, code 4+p): pairs 0,1 at fraction bits 4-7 (1024 + 16q), pairs 2,3
// at bits 6-9 (1024 + 64q).  Three shifts + four and-or.
__device__ __forceinline__ void extract_w4(uint32_t w, uint32_t e[4], uint32_t mv) {
    e[0] = magic(w << 4, 0x00F000F0u, mv);
    e[1] = magic(w, 0x00F000F0u, mv);
    e[2] = magic(w >> 2, 0x03C003C0u, mv);
    e[3] = magic(w >> 6, 0x03C003C0u, mv);
}

// 16^-1 / 64^-1 for the 4-bit pair positions above.
__device__ __forceinline__ float w4_pair_scale(int p) { return p < 2 ? 1.0f / 16 : 1.0f / 64; }

// Opaque identity: the value is treated as redefined here, so work derived
// from registers preloaded before a loop is not hoisted out of the loop
// (which would keep every unpacked code live at once).
__device__ __forceinline__ void pin(uint32_t& v) { __asm__ volatile("" : "+v"(v)); }
// The four words of v are materialized here: the loads that produce them
// complete before this point, later loads stay in flight.
__device__ __forceinline__ void pin4(uint4& v) {
    __asm__ volatile("" : "+v"(v.x), "+v"(v.y), "+v"(v.z), "+v"(v.w));
}

// Wait until at most N vector-memory loads of this wave are outstanding
// (s_waitcnt vmcnt(N); expcnt and lgkmcnt are left alone).  Used to bound
// the loads a wave keeps in flight while it streams weights, so that the
// memory queues stay short and the small hand-off messages of the other
// compute units are not queued behind the whole stream.
template <int N>
__device__ __forceinline__ void vm_window() {
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Lane permutations within rows of 16 lanes (DPP, no LDS round trip).
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                                  0xF, 0xF, false));
}
constexpr int DPP_QUAD_XOR1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int DPP_QUAD_XOR2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141;  // lane i <- lane 7 - i within 8
constexpr int DPP_MIRROR = 0x140;       // lane i <- lane 15 - i within 16

// Sum over the WIDTH consecutive lanes sharing an output row (every lane of
// the group ends with the total).  Within 16 lanes the steps are DPP moves
// (two quad swaps, then the mirrors, which pair each lane with one of the
// other half once every half holds its own sum); wider groups add xor
// shuffles across rows.
template <int WIDTH>
__device__ __forceinline__ float group_sum(float v) {
    if constexpr (WIDTH >= 2) v += dpp<DPP_QUAD_XOR1>(v);
    if constexpr (WIDTH >= 4) v += dpp<DPP_QUAD_XOR2>(v);
    if constexpr (WIDTH >= 8) v += dpp<DPP_HALF_MIRROR>(v);
    if constexpr (WIDTH >= 16) v += dpp<DPP_MIRROR>(v);
    if constexpr (WIDTH >= 32) v += __shfl_xor(v, 16, 64);
    if constexpr (WIDTH >= 64) v += __shfl_xor(v, 32, 64);
    return v;
}

}  // namespace qmlp

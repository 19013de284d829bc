// Launch-shape helpers shared by the decode kernels' host launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace qmlp {

inline int mtile_for(int M) { return M <= 1 ? 1 : M <= 2 ? 2 : M <= 4 ? 4 : M <= 8 ? 8 : 16; }

// Lanes per row: as few as keep every lane's unit count within MAXJ = 16.
inline int lanes_gateup(int U) { return U <= 128 ? 8 : U <= 256 ? 16 : U <= 512 ? 32 : 64; }
inline int lanes_down(int U) { return U <= 64 ? 8 : U <= 128 ? 16 : U <= 256 ? 32 : 64; }
inline int maxj_for(int J) { return J <= 8 ? 8 : 16; }
// Lanes per row for 16-byte units of `bits`-bit codes (64 codes per unit at
// 2 bits, 32 at 4 bits): each width keeps the policy of its own unit size.
inline int lanes_for(int U, int bits) { return bits == 4 ? lanes_down(U) : lanes_gateup(U); }

// The fewest lanes per row that keep every lane within 16 units: the most
// loads in flight per lane, for launches whose parallelism comes from many
// blocks (batches).
inline int lanes_fewest(int U) { return U <= 128 ? 8 : U <= 256 ? 16 : U <= 512 ? 32 : 64; }
inline bool units_fit(int k, int bits) {
    const int U = k / codes_per_unit(bits);
    const int S = lanes_for(U, bits);
    return (U + S - 1) / S <= 16;
}

constexpr int kLdsBudget = 64 * 1024;

template <typename K>
inline hipError_t set_lds(K kernel, size_t bytes) {
    if (bytes <= 64 * 1024)
        return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

inline int units_per_chunk(int U, int S, size_t bytes_per_unit_token, int mt) {
    long uc = (long)(kLdsBudget / (bytes_per_unit_token * (size_t)mt));
    uc = uc / S * S;
    if (uc < S) uc = S;
    if (uc > U) uc = (U + S - 1) / S * S;
    return (int)uc;
}

inline bool decode_shape_supported_impl(int d, int f) {
    const int Ug = d / 64, Ud = f / 32;
    return (Ug + lanes_gateup(Ug) - 1) / lanes_gateup(Ug) <= 16 &&
           (Ud + lanes_down(Ud) - 1) / lanes_down(Ud) <= 16;
}

}  // namespace qmlp

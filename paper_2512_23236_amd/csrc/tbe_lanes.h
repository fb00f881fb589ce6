// Lane exchanges within a wave (gfx950) that do not go through the LDS, and
// the group sums built from them.

#pragma once

#include <hip/hip_runtime.h>

namespace tbe {

// x of lane v ^ D (D a power of two below 64) without the LDS: inside a
// 16-lane row by DPP moves (quad permutations for 1 and 2; row rotations
// otherwise: by 8 it is the xor, and distance 4 picks the rotation by 4 or by
// 12 by the lane's bit 2); across rows by the gfx950 lane-swap instructions,
// whose two results hold, for every lane, the values of both lanes of its
// pair (the lower lane's first).
template <int D>
__device__ inline float xor_lane(float x, int v) {
    const int xi = __float_as_int(x);
    if constexpr (D == 1) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(xi, 0xB1, 0xF, 0xF, false));  // quad_perm [1,0,3,2]
    } else if constexpr (D == 2) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(xi, 0x4E, 0xF, 0xF, false));  // quad_perm [2,3,0,1]
    } else if constexpr (D == 4) {
        const int a = __builtin_amdgcn_mov_dpp(xi, 0x124, 0xF, 0xF, false);  // row_ror:4
        const int b = __builtin_amdgcn_mov_dpp(xi, 0x12C, 0xF, 0xF, false);  // row_ror:12
        return __int_as_float((v & 4) ? a : b);
    } else if constexpr (D == 8) {
        return __int_as_float(__builtin_amdgcn_mov_dpp(xi, 0x128, 0xF, 0xF, false));  // row_ror:8
    } else if constexpr (D == 16) {
        const auto p = __builtin_amdgcn_permlane16_swap(static_cast<unsigned>(xi), static_cast<unsigned>(xi), false,
                                                        false);
        return __uint_as_float((v & 16) ? p[0] : p[1]);
    } else {
        static_assert(D == 32, "distance");
        const auto p = __builtin_amdgcn_permlane32_swap(static_cast<unsigned>(xi), static_cast<unsigned>(xi), false,
                                                        false);
        return __uint_as_float((v & 32) ? p[0] : p[1]);
    }
}

// Sum of x over the lanes of the group holding lane v, from distance D down
// to 1 (a group of 2D lanes), by a butterfly in a fixed order (every lane of
// the group gets the same sum).
template <int D>
__device__ inline float xsum_from(float x, int v) {
    if constexpr (D >= 1) return xsum_from<D / 2>(x + xor_lane<D>(x, v), v);
    else return x;
}

// Sum of x over the LPR lanes of the group holding lane v (lanes sharing
// v / LPR).
template <int LPR>
__device__ inline float group_xsum(float x, int v) {
    return xsum_from<LPR / 2>(x, v);
}

}  // namespace tbe

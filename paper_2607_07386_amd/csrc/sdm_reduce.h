// Cross-lane sums for the backward scan (gfx950, wave64).
#pragma once

#include "sdm_common.h"

namespace sdm_reduce {

// Lane (this lane ^ M) for M <= 8 through a DPP row/quad permute with a zero
// "old" value and bound_ctrl: every lane reads in range, so the value is the
// same as a plain permute, and the compiler can fold the permute into the
// VALU op that consumes it (v_add_f32_dpp) instead of a separate move.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
template <int M>
__device__ __forceinline__ float xor_dpp(float v) {
    static_assert(M == 1 || M == 2 || M == 4 || M == 8, "DPP distances within a row");
    if constexpr (M == 1) return dpp_f<0xB1>(v);              // quad_perm [1,0,3,2]
    else if constexpr (M == 2) return dpp_f<0x4E>(v);         // quad_perm [2,3,0,1]
    else if constexpr (M == 4) return dpp_f<0x1B>(dpp_f<0x141>(v));   // row_half_mirror (i ^ 7), quad_perm [3,2,1,0] (^ 3)
    else return dpp_f<0x128>(v);                              // row_ror:8
}

// v plus the value of lane (this lane ^ M), the same in both lanes of a pair.
// For M = 16, 32 a permlane swap of v with itself leaves one side of each
// pair in one result and the other side in the other: their sum is the pair
// sum in every lane, with no lane select.
template <int M>
__device__ __forceinline__ float add_xor(float v) {
    const uint32_t u = __float_as_uint(v);
    if constexpr (M == 32) {
        const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        return __uint_as_float(r[0]) + __uint_as_float(r[1]);
    } else if constexpr (M == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
        return __uint_as_float(r[0]) + __uint_as_float(r[1]);
    } else {
        return v + xor_dpp<M>(v);
    }
}
// Sum over xor distances M0, 2 M0, ..., 8 (within a 16-lane row).
template <int M0>
__device__ __forceinline__ float row_sum_from(float v) {
    if constexpr (M0 >= 16) return v;
    else return row_sum_from<M0 * 2>(add_xor<M0>(v));
}
// Sum over all 64 lanes, every lane receiving it.
__device__ __forceinline__ float wave_sum(float v) {
    return add_xor<32>(add_xor<16>(row_sum_from<1>(v)));
}

namespace detail {
__device__ __forceinline__ float swap32_sum(float lo_src, float hi_src) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(lo_src), __float_as_uint(hi_src), false,
                                                    false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float swap16_sum(float a, float b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
// z holds one value per 16-lane row, [A B C D]; out[r] = row r's value in every lane.
__device__ __forceinline__ void rows_gather4(float z, float (&out)[4]) {
    const auto h = __builtin_amdgcn_permlane32_swap(__float_as_uint(z), __float_as_uint(z), false,
                                                    false);                       // [A B A B], [C D C D]
    const auto s = __builtin_amdgcn_permlane16_swap(h[0], h[0], false, false);   // [A A A A], [B B B B]
    const auto t = __builtin_amdgcn_permlane16_swap(h[1], h[1], false, false);   // [C C C C], [D D D D]
    out[0] = __uint_as_float(s[0]);
    out[1] = __uint_as_float(s[1]);
    out[2] = __uint_as_float(t[0]);
    out[3] = __uint_as_float(t[1]);
}
}  // namespace detail

// For the eight floats of a and b: the sum over the lanes of this lane's
// class (lane % CQ), in every lane.  Reduce-scatter first: a permlane32 swap
// of two values then an add leaves one value's half-sums in the lower 32
// lanes and the other's in the upper 32, and a permlane16 swap does the same
// across 16-lane rows, so every add step halves the registers in play (8 -> 4
// -> 2).  Then butterflies within a row over the distances CQ .. 8, then an
// all-gather by swapping each register with a copy of itself.  32 VALU
// instructions at CQ = 2, against 14 per float for independent butterflies.
template <int CQ>
__device__ __forceinline__ void rows_allreduce8(v4f& a, v4f& b) {
    static_assert(CQ >= 1 && CQ <= 8 && (CQ & (CQ - 1)) == 0, "class count must divide a row");
    const float y0 = detail::swap32_sum(a.x, b.x);   // halves [a.x | b.x]
    const float y1 = detail::swap32_sum(a.y, b.y);
    const float y2 = detail::swap32_sum(a.z, b.z);
    const float y3 = detail::swap32_sum(a.w, b.w);
    float z0 = detail::swap16_sum(y0, y2);           // rows [a.x a.z b.x b.z]
    float z1 = detail::swap16_sum(y1, y3);           // rows [a.y a.w b.y b.w]
    z0 = row_sum_from<CQ>(z0);
    z1 = row_sum_from<CQ>(z1);
    float o0[4], o1[4];
    detail::rows_gather4(z0, o0);
    detail::rows_gather4(z1, o1);
    a = v4f{o0[0], o1[0], o0[1], o1[1]};
    b = v4f{o0[2], o1[2], o0[3], o1[3]};
}

// The sum of v over the lanes of this lane's class (lane % CQ), in every lane.
template <int CQ>
__device__ __forceinline__ float class_sum(float v) {
    return add_xor<32>(add_xor<16>(row_sum_from<CQ>(v)));
}

// Same for the four floats of one v4f (16 VALU instructions at CQ = 2).
template <int CQ>
__device__ __forceinline__ void rows_allreduce4(v4f& a) {
    static_assert(CQ >= 1 && CQ <= 8 && (CQ & (CQ - 1)) == 0, "class count must divide a row");
    const float y0 = detail::swap32_sum(a.x, a.z);   // halves [x | z]
    const float y1 = detail::swap32_sum(a.y, a.w);   // halves [y | w]
    float z = detail::swap16_sum(y0, y1);            // rows [x y z w]
    z = row_sum_from<CQ>(z);
    float o[4];
    detail::rows_gather4(z, o);
    a = v4f{o[0], o[1], o[2], o[3]};
}

}  // namespace sdm_reduce

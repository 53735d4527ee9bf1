// Wavefront reductions for wave64 on gfx950.
//
// Steps inside a 16-lane row use DPP (quad_perm, row_half_mirror, row_ror),
// which are plain VALU operands instead of LDS permutes; only the two steps
// that cross rows go through ds_swizzle/bpermute.  Every lane of a group ends
// with the same value: each step combines a lane with a partner that holds
// the mirrored partial, and IEEE add/max are commutative.
#pragma once

#include <hip/hip_runtime.h>

namespace mtp {

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, false);
}

constexpr int DPP_XOR1 = 0xB1;          // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4E;          // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141;  // lane i <-> 7 - i within each 8 lanes
constexpr int DPP_ROR8 = 0x128;         // rotate a 16-lane row by 8

// Sum over each aligned group of 8 lanes.
__device__ __forceinline__ float sum8(float v) {
    v += dpp_f<DPP_XOR1>(v);
    v += dpp_f<DPP_XOR2>(v);
    v += dpp_f<DPP_HALF_MIRROR>(v);
    return v;
}
__device__ __forceinline__ float sum16(float v) {
    v = sum8(v);
    v += dpp_f<DPP_ROR8>(v);
    return v;
}
// Combine each lane's value with that of the lane 16 (32) apart without an
// LDS round trip: the gfx950 permlane swaps of a value with itself give every
// lane its row pair's lower and upper values (r[0], r[1]), and add / max are
// commutative, so both partner lanes get the bit-identical result a shuffle
// would give.
__device__ __forceinline__ float pl_lo16(float v, float& hi) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    hi = __uint_as_float(r[1]);
    return __uint_as_float(r[0]);
}
__device__ __forceinline__ float pl_lo32(float v, float& hi) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    hi = __uint_as_float(r[1]);
    return __uint_as_float(r[0]);
}
__device__ __forceinline__ float xor16_sum(float v) { float h; const float l = pl_lo16(v, h); return l + h; }
__device__ __forceinline__ float xor32_sum(float v) { float h; const float l = pl_lo32(v, h); return l + h; }
__device__ __forceinline__ float xor16_max(float v) { float h; const float l = pl_lo16(v, h); return fmaxf(l, h); }
__device__ __forceinline__ float xor32_max(float v) { float h; const float l = pl_lo32(v, h); return fmaxf(l, h); }

__device__ __forceinline__ float wave_sum64(float v) {
    v = sum16(v);
    v = xor16_sum(v);
    v = xor32_sum(v);
    return v;
}
__device__ __forceinline__ float max16(float v) {
    v = fmaxf(v, dpp_f<DPP_XOR1>(v));
    v = fmaxf(v, dpp_f<DPP_XOR2>(v));
    v = fmaxf(v, dpp_f<DPP_HALF_MIRROR>(v));
    v = fmaxf(v, dpp_f<DPP_ROR8>(v));
    return v;
}
__device__ __forceinline__ float wave_max64(float v) {
    v = max16(v);
    v = xor16_max(v);
    v = xor32_max(v);
    return v;
}
// Sum over lanes that are 8, 16 and 32 apart (lanes with equal lane % 8).
__device__ __forceinline__ float sum_stride8(float v) {
    v += dpp_f<DPP_ROR8>(v);
    v = xor16_sum(v);
    v = xor32_sum(v);
    return v;
}

// (value, index) maximum over the wave under the total order "larger value,
// then smaller index"; every lane ends with the winner.
// (value, index) order: larger value first, lower index on ties.  Written
// with bitwise ops and selects so that no step becomes a branch.
__device__ __forceinline__ bool vi_better(float va, int ia, float vb, int ib) {
    return (va > vb) | ((va == vb) & (ia < ib));
}
template <int CTRL>
__device__ __forceinline__ void vi_step_dpp(float& v, int& i) {
    const float ov = dpp_f<CTRL>(v);
    const int oi = dpp_i<CTRL>(i);
    const bool b = vi_better(ov, oi, v, i);
    v = b ? ov : v;
    i = b ? oi : i;
}
__device__ __forceinline__ void vi_step_shfl(float& v, int& i, int mask) {
    const float ov = __shfl_xor(v, mask);
    const int oi = __shfl_xor(i, mask);
    const bool b = vi_better(ov, oi, v, i);
    v = b ? ov : v;
    i = b ? oi : i;
}
// Every lane ends with the wave's best (value, index).
__device__ __forceinline__ void wave_argmax(float& v, int& i) {
    vi_step_dpp<DPP_XOR1>(v, i);
    vi_step_dpp<DPP_XOR2>(v, i);
    vi_step_dpp<DPP_HALF_MIRROR>(v, i);
    vi_step_dpp<DPP_ROR8>(v, i);
    vi_step_shfl(v, i, 16);
    vi_step_shfl(v, i, 32);
}

// The wave's best (value, index) as uniform values, crossing rows with DPP
// row broadcasts (lane 15 -> rows 1 and 3, lane 31 -> rows 2 and 3) so that
// lane 63 ends with the result; no LDS permute on the way.
template <int CTRL, int ROWS>
__device__ __forceinline__ void vi_step_bcast(float& v, int& i) {
    const float ov = __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(v), __float_as_int(v), CTRL, ROWS, 0xF, false));
    const int oi = __builtin_amdgcn_update_dpp(i, i, CTRL, ROWS, 0xF, false);
    const bool b = vi_better(ov, oi, v, i);
    v = b ? ov : v;
    i = b ? oi : i;
}
__device__ __forceinline__ void wave_argmax_uniform(float& v, int& i) {
    vi_step_dpp<DPP_XOR1>(v, i);
    vi_step_dpp<DPP_XOR2>(v, i);
    vi_step_dpp<DPP_HALF_MIRROR>(v, i);
    vi_step_dpp<DPP_ROR8>(v, i);
    vi_step_bcast<0x142, 0xA>(v, i);   // row_bcast:15 into rows 1, 3
    vi_step_bcast<0x143, 0xC>(v, i);   // row_bcast:31 into rows 2, 3
    v = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
    i = __builtin_amdgcn_readlane(i, 63);
}

}  // namespace mtp

// Reductions across the lanes of a 64-lane wavefront without LDS: DPP inside
// 16-lane rows (quad_perm and the row mirrors), then the gfx950 row swaps
// (v_permlane16_swap, v_permlane32_swap) across rows. Every step combines a
// lane with a partner that combines it back in the other order, so for a
// commutative operation all lanes involved end with the same bits.
#pragma once

#include <hip/hip_runtime.h>

namespace tx {

constexpr int kDppQuadXor1 = 0xB1;       // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4E;       // quad_perm [2, 3, 0, 1]
constexpr int kDppRowHalfMirror = 0x141;  // lane i of 8 reads lane 7 - i
constexpr int kDppRowMirror = 0x140;      // lane i of 16 reads lane 15 - i

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// With two copies of x, v_permlane32_swap leaves (x[l mod 32], x[32 + l mod 32])
// in its two results on lane l, v_permlane16_swap the values of the two
// 16-lane rows of l's pair of rows (0-1 or 2-3).
__device__ __forceinline__ float xor32_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float row16_sum(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float row16_max(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Sum over each group of 4 lanes (l ^ 1, l ^ 2).
__device__ __forceinline__ float quad_sum(float x) {
  x += dpp_f32<kDppQuadXor1>(x);
  return x + dpp_f32<kDppQuadXor2>(x);
}

// Sum and maximum over the whole wavefront, on every lane.
__device__ __forceinline__ float wave_sum(float x) {
  x = quad_sum(x);
  x += dpp_f32<kDppRowHalfMirror>(x);
  x += dpp_f32<kDppRowMirror>(x);
  return xor32_sum(row16_sum(x));
}
__device__ __forceinline__ float wave_max(float x) {
  x = fmaxf(x, dpp_f32<kDppQuadXor1>(x));
  x = fmaxf(x, dpp_f32<kDppQuadXor2>(x));
  x = fmaxf(x, dpp_f32<kDppRowHalfMirror>(x));
  x = fmaxf(x, dpp_f32<kDppRowMirror>(x));
  return xor32_max(row16_max(x));
}

}  // namespace tx

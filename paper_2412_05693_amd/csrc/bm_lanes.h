// Cross-lane reductions in registers for the decode kernels (gfx950, wave64).
//
// Quad permutes for lanes 1 and 2 apart and the mirrored halves of each 8- and
// 16-lane row (DPP), a rotation by 8 inside a 16-lane row, and gfx950's swaps
// of the 16- and 32-lane halves of a wave replace LDS shuffles (ds_bpermute):
// no LDS round trip per step.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace bm {
namespace lanes {

// Wave-wide reductions: each step combines two disjoint lane groups that
// already agree on their own result, so every lane ends with the wave's.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t x) {
  return __builtin_amdgcn_update_dpp(x, x, CTRL, 0xF, 0xF, false);
}

template <typename Op>
__device__ __forceinline__ uint32_t wave_reduce(uint32_t x, Op op) {
  x = op(x, dpp<0xB1>(x));    // quad_perm [1,0,3,2]
  x = op(x, dpp<0x4E>(x));    // quad_perm [2,3,0,1]
  x = op(x, dpp<0x141>(x));   // row_half_mirror
  x = op(x, dpp<0x140>(x));   // row_mirror
  const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = op(a[0], a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return op(b[0], b[1]);
}

__device__ __forceinline__ float wave_max(float v) {
  return __uint_as_float(wave_reduce(__float_as_uint(v), [](uint32_t a, uint32_t b) {
    return __float_as_uint(fmaxf(__uint_as_float(a), __uint_as_float(b)));
  }));
}

__device__ __forceinline__ float wave_sum(float v) {
  return __uint_as_float(wave_reduce(__float_as_uint(v), [](uint32_t a, uint32_t b) {
    return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
  }));
}

// v plus the value of the lane OFF apart (lane ^ OFF) for OFF = 8, 16, 32: a
// row rotation by 8 inside each 16-lane row, gfx950's half swaps for 16 and 32
template <int OFF>
__device__ __forceinline__ float add_xor(float v) {
  const uint32_t x = __float_as_uint(v);
  if constexpr (OFF == 8) {
    return v + __uint_as_float(dpp<0x128>(x));   // row_ror:8
  } else if constexpr (OFF == 16) {
    const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    return __uint_as_float(a[0]) + __uint_as_float(a[1]);
  } else {
    static_assert(OFF == 32, "lane offsets 8, 16 or 32");
    const auto a = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return __uint_as_float(a[0]) + __uint_as_float(a[1]);
  }
}

// smallest 64-bit key of the wave (the same steps on both halves of the key)
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t k) {
  uint32_t lo = (uint32_t)k, hi = (uint32_t)(k >> 32);
  auto take = [&](uint32_t plo, uint32_t phi) {
    if ((((uint64_t)phi << 32) | plo) < (((uint64_t)hi << 32) | lo)) {
      lo = plo;
      hi = phi;
    }
  };
  take(dpp<0xB1>(lo), dpp<0xB1>(hi));
  take(dpp<0x4E>(lo), dpp<0x4E>(hi));
  take(dpp<0x141>(lo), dpp<0x141>(hi));
  take(dpp<0x140>(lo), dpp<0x140>(hi));
  {
    const auto a = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto b = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    lo = a[0];
    hi = b[0];
    take(a[1], b[1]);
  }
  {
    const auto a = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
    const auto b = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
    lo = a[0];
    hi = b[0];
    take(a[1], b[1]);
  }
  return ((uint64_t)hi << 32) | lo;
}

// Sum over each group of N consecutive lanes (N a power of two, 2 to 32), every
// lane of the group receiving it: the first steps of the wave-wide reduction
// (the same additions as a butterfly over lanes 1, 2, 4, ... apart).
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(N == 2 || N == 4 || N == 8 || N == 16 || N == 32, "group of 2 to 32 lanes");
  uint32_t x = __float_as_uint(v);
  auto add = [](uint32_t a, uint32_t b) { return __float_as_uint(__uint_as_float(a) + __uint_as_float(b)); };
  x = add(x, dpp<0xB1>(x));
  if constexpr (N >= 4) x = add(x, dpp<0x4E>(x));
  if constexpr (N >= 8) x = add(x, dpp<0x141>(x));
  if constexpr (N >= 16) x = add(x, dpp<0x140>(x));
  if constexpr (N >= 32) {
    const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    x = add(a[0], a[1]);
  }
  return __uint_as_float(x);
}

}  // namespace lanes
}  // namespace bm

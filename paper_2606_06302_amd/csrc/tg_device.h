// Device-side helpers for the gfx950 kernels of libtangram.so.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace tgd {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }

// fp32 -> bf16 bits, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// a.lo*b.lo + a.hi*b.hi + c on packed bf16 pairs, fp32 accumulate.
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// DPP lane movement inside 16-lane rows.
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
constexpr int kQuadXor1 = 0xB1;       // quad_perm [1,0,3,2]
constexpr int kQuadXor2 = 0x4E;       // quad_perm [2,3,0,1]
constexpr int kRowHalfMirror = 0x141; // lane i <- 7-i inside each 8-lane half row
constexpr int kRowMirror = 0x140;     // lane i <- 15-i inside each row
constexpr int kRowRor8 = 0x128;       // lane i <- (i+8) mod 16 inside each row

// Sum over aligned groups of N lanes (N in {1, 2, 4, 8, 16}); every lane of
// the group receives the group total.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
  if constexpr (N >= 2) x += dpp<kQuadXor1>(x);
  if constexpr (N >= 4) x += dpp<kQuadXor2>(x);
  if constexpr (N >= 8) x += dpp<kRowHalfMirror>(x);
  if constexpr (N >= 16) x += dpp<kRowMirror>(x);
  return x;
}

// Combination across the 16-lane rows of a wave: lanes l and l^16 (swap16)
// and lanes l and l^32 (swap32), using the gfx950 permlane swaps.
__device__ __forceinline__ float swap16_sum(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float swap32_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float swap16_max(float x) {
  auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float swap32_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Reduction over the token rows of a wave whose rows are ROWLANES lanes wide
// (ROWLANES in {8, 16, 32}): every lane receives the total over the
// 64/ROWLANES lanes that share its position within a row.
template <int ROWLANES>
__device__ __forceinline__ float rows_sum(float x) {
  if constexpr (ROWLANES <= 8) x += dpp<kRowRor8>(x);
  if constexpr (ROWLANES <= 16) x = swap16_sum(x);
  return swap32_sum(x);
}
template <int ROWLANES>
__device__ __forceinline__ float rows_max(float x) {
  if constexpr (ROWLANES <= 8) x = fmaxf(x, dpp<kRowRor8>(x));
  if constexpr (ROWLANES <= 16) x = swap16_max(x);
  return swap32_max(x);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace tgd

// Internal device helpers shared by the HIP kernels of libspexis (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spexis {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }

// 16-byte global load / store (the address must be 16-byte aligned).
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// fp32 -> bf16 bits, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint32_t bf16_bits(float x) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(x)));
}
// Two values in one v_cvt_pk_bf16_f32 (the same rounding as bf16_bits; converting them one at a
// time costs a shift and a merge per pair on top).
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2 f = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// DPP lane controls: row_shr:n (n = 1..15), broadcast of lane 15 of each row into the next
// row, broadcast of lane 31 into rows 2 and 3, and quad permutations.
constexpr int kDppRowShr = 0x110;
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;
constexpr int kDppQuadXor1 = 0xB1;   // quad_perm [1, 0, 3, 2]
constexpr int kDppQuadXor2 = 0x4E;   // quad_perm [2, 3, 0, 1]
// Inclusive prefix sum over the lanes of a wave, in DPP moves only (no LDS round trips):
// shifts by 1, 2, 4 and 8 within each row of 16 lanes (lanes shifted in from outside the row
// add 0), then row r adds the total of row r-1 (rows 1, 3) and rows 2, 3 add lane 31.
__device__ __forceinline__ int wave_incl_scan_i32(int v, int lane) {
  (void)lane;
  v += __builtin_amdgcn_update_dpp(0, v, kDppRowShr + 1, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, kDppRowShr + 2, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, kDppRowShr + 4, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, kDppRowShr + 8, 0xF, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, kDppRowBcast15, 0xA, 0xF, false);
  v += __builtin_amdgcn_update_dpp(0, v, kDppRowBcast31, 0xC, 0xF, false);
  return v;
}
// Sum over the lanes of a wave (the same value in every lane).
__device__ __forceinline__ int wave_sum_i32(int v) {
  return __builtin_amdgcn_readlane(wave_incl_scan_i32(v, 0), kWave - 1);
}
// A DPP lane move of a 32-bit value; lanes the move does not write get `old`.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v, uint32_t old) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, kCtrl, kRowMask, 0xF, false);
}
// Reductions over the 64 lanes of a wave, in DPP moves (the pattern of the integer scan, so lane
// 63 ends with the whole wave's result), broadcast with readlane: the result is uniform.
#define SPEXIS_DPP_REDUCE(v, move, op) \
  v = op(v, move<kDppRowShr + 1, 0xF>(v));     \
  v = op(v, move<kDppRowShr + 2, 0xF>(v));     \
  v = op(v, move<kDppRowShr + 4, 0xF>(v));     \
  v = op(v, move<kDppRowShr + 8, 0xF>(v));     \
  v = op(v, move<kDppRowBcast15, 0xA>(v));     \
  v = op(v, move<kDppRowBcast31, 0xC>(v));

template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_max_move(float v) {
  return __uint_as_float(dpp_u32<kCtrl, kRowMask>(__float_as_uint(v), 0xFF800000u));   // -inf elsewhere
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_sum_move(float v) {
  return __uint_as_float(dpp_u32<kCtrl, kRowMask>(__float_as_uint(v), 0u));
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int dpp_or_move(int v) {
  return (int)dpp_u32<kCtrl, kRowMask>((uint32_t)v, 0u);
}
template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint64_t dpp_u64_move(uint64_t v) {
  const uint32_t lo = dpp_u32<kCtrl, kRowMask>((uint32_t)v, 0u);
  const uint32_t hi = dpp_u32<kCtrl, kRowMask>((uint32_t)(v >> 32), 0u);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ float op_max(float a, float b) { return fmaxf(a, b); }
__device__ __forceinline__ float op_addf(float a, float b) { return a + b; }
__device__ __forceinline__ int op_or(int a, int b) { return a | b; }
__device__ __forceinline__ uint64_t op_addu64(uint64_t a, uint64_t b) { return a + b; }

__device__ __forceinline__ float readlane_f32(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}
__device__ __forceinline__ uint64_t readlane_u64(uint64_t v, int lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), lane);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ float wave_max(float v) {
  SPEXIS_DPP_REDUCE(v, dpp_max_move, op_max)
  return readlane_f32(v, kWave - 1);
}
// (the summation order is fixed: every caller of wave_sum on the same values gets the same sum)
__device__ __forceinline__ float wave_sum(float v) {
  SPEXIS_DPP_REDUCE(v, dpp_sum_move, op_addf)
  return readlane_f32(v, kWave - 1);
}
__device__ __forceinline__ int wave_or(int v) {
  SPEXIS_DPP_REDUCE(v, dpp_or_move, op_or)
  return __builtin_amdgcn_readlane(v, kWave - 1);
}
// Inclusive prefix sum of 64-bit values over the lanes of a wave, and the wave's total.
__device__ __forceinline__ uint64_t wave_incl_scan_u64(uint64_t v) {
  SPEXIS_DPP_REDUCE(v, dpp_u64_move, op_addu64)
  return v;
}
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) { return readlane_u64(wave_incl_scan_u64(v), kWave - 1); }

}  // namespace spexis

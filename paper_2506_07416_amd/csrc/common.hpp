// Device-side helpers shared by the LiteVLM kernels (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace litevlm {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;

// fp32 -> bf16 bits, round to nearest even (inputs here are finite).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// Pack 8 fp32 into one MFMA bf16x8 operand (round to nearest even).
__device__ __forceinline__ bf16x8 pack_bf16x8(const float* x) {
  i32x4 w;
  w[0] = (int)(f32_to_bf16_bits(x[0]) | ((uint32_t)f32_to_bf16_bits(x[1]) << 16));
  w[1] = (int)(f32_to_bf16_bits(x[2]) | ((uint32_t)f32_to_bf16_bits(x[3]) << 16));
  w[2] = (int)(f32_to_bf16_bits(x[4]) | ((uint32_t)f32_to_bf16_bits(x[5]) << 16));
  w[3] = (int)(f32_to_bf16_bits(x[6]) | ((uint32_t)f32_to_bf16_bits(x[7]) << 16));
  return __builtin_bit_cast(bf16x8, w);
}

__device__ __forceinline__ float wave_max_xor(float x, int lanemask) {
  return fmaxf(x, __shfl_xor(x, lanemask, kWave));
}

// Cross-row exchanges on the gfx950 permlane swaps: the pair returned holds
// {x[lane], x[lane ^ 16]} (resp. ^ 32) with the lower row first in both lanes,
// so a sum of the pair is bitwise identical in the two lanes.
__device__ __forceinline__ float2 pair_xor16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float2 pair_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return make_float2(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor16(float x) { const float2 p = pair_xor16(x); return fmaxf(p.x, p.y); }
__device__ __forceinline__ float max_xor32(float x) { const float2 p = pair_xor32(x); return fmaxf(p.x, p.y); }
__device__ __forceinline__ float sum_xor16(float x) { const float2 p = pair_xor16(x); return p.x + p.y; }
__device__ __forceinline__ float sum_xor32(float x) { const float2 p = pair_xor32(x); return p.x + p.y; }

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
// Sum over each row of 16 lanes (xor 1, xor 2, half-mirror, mirror); every
// lane of the row ends with the same bits.
__device__ __forceinline__ float row16_sum(float x) {
  x += dpp<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp<0x141>(x);  // row_half_mirror
  x += dpp<0x140>(x);  // row_mirror
  return x;
}

// OCP E4M3FN byte -> fp32 (exact). Used only where an fp8 operand must be
// widened for a non-MFMA step.
__device__ __forceinline__ float e4m3_to_f32(uint32_t b) {
  uint32_t s = (b >> 7) & 1u, e = (b >> 3) & 0xFu, m = b & 7u;
  float mag;
  if (e == 0u) mag = (float)m * 0.001953125f;  // m/8 * 2^-6
  else mag = __uint_as_float(((e + 120u) << 23) | (m << 20));
  if (e == 15u && m == 7u) mag = __uint_as_float(0x7FC00000u);
  return s ? -mag : mag;
}

}  // namespace litevlm

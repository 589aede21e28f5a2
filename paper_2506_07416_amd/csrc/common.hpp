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

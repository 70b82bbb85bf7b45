// Device helpers shared by the gfx950 kernels: vector types, matrix-core
// wrappers, bf16 / fp16 conversions and wavefront reductions.
//
// Matrix-core lane layout used throughout (64-lane wavefront, lane l,
// group G = l / 16, column c = l % 16), for D[16x16] += A[16xK] * B[Kx16]:
//   A operand: lane l holds A[c][K-slice of group G]
//   B operand: lane l holds B[K-slice of group G][c]
//   accumulator: lane l holds D[4G + i][c], i = 0..3
// Any assignment of the K index to (G, element) is valid as long as A and B
// use the same one; the kernels exploit that freedom to read contiguous
// memory.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sd {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4;

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ floatx4 mfma_bf16(const bf16x8& a, const bf16x8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_f16(const f16x8& a, const f16x8& b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mfma_f32(float a, float b, const floatx4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// bf16 bit pattern <-> float (exact widening; narrowing rounds to nearest even)
__device__ __forceinline__ float bf16_bits_to_float(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

__device__ __forceinline__ __bf16 float_to_bf16(float x) {
  return (__bf16)x;   // round to nearest even
}

__device__ __forceinline__ float bf16_to_float(__bf16 x) {
  return (float)x;
}

// 16-byte vector of 8 bf16 values viewed as raw words
union Pack8 {
  uint4 u;
  bf16x8 b;
  f16x8 h;
  uint16_t s[8];
};

__device__ __forceinline__ float wave_max_across_groups(float v) {
  // reduce over lanes l, l^16, l^32, l^48 (same column, four groups)
  v = fmaxf(v, __shfl_xor(v, 16, 64));
  v = fmaxf(v, __shfl_xor(v, 32, 64));
  return v;
}

__device__ __forceinline__ float wave_sum_across_groups(float v) {
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}

}  // namespace sd

// Shared device helpers for the SAO kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sao {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
// 16-byte chunk as a native vector: copies lower to plain vector loads/stores
// (HIP's uint4 is a struct whose copies become memcpy through private memory).
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

// Storage type tags for the head operands.
struct BF16 {
  using storage = uint16_t;
  static constexpr int kPerChunk = 8;  // elements per 16-byte chunk
};
struct F32 {
  using storage = float;
  static constexpr int kPerChunk = 4;
};

// Two floats as packed bf16, rounded to nearest even (gfx950's
// v_cvt_pk_bf16_f32; NaN stays NaN): `lo` in bits 0-15, `hi` in bits 16-31.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {static_cast<__bf16>(lo), static_cast<__bf16>(hi)};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ int64_t round_up_dev(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Merge two (max, sum of exp(x - max)) pairs of one log-sum-exp.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -__builtin_inff()) return;  // both empty
  s = s * fast_exp2((m - mn) * kLog2e) + s2 * fast_exp2((m2 - mn) * kLog2e);
  m = mn;
}

template <typename T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

}  // namespace sao

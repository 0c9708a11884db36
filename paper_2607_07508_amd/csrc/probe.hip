// Measurement probe, not part of the SAO pass (built into libsao_probe.so, loaded
// only by the benchmark's --mfma-ceiling mode): how fast the bf16 MFMA pipe runs
// on this chip with nothing but MFMAs to issue, in the head kernels' arrangement
// (one wave per SIMD, 4 x 4 blocks of v_mfma_f32_32x32x16_bf16 on 256
// accumulator registers, 8 operand fragments), for operand data of different
// bit activity. The clock drops with the switching activity of the operands, so
// this bounds what any bf16 kernel can reach on real data.
//
// mode 0: random bf16 operands (N(0, 1)-like bit patterns), fixed per wave
// mode 1: constant operands (every element 1.0)
// mode 2: random operands whose A fragments get new bits every iteration (a few
//         VALU operations per dword, issued between the MFMAs), so that the
//         MFMAs keep seeing fresh operand bits as in a real K loop
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t mix(uint32_t x) {
  x ^= x >> 16;
  x *= 0x7feb352dU;
  x ^= x >> 15;
  x *= 0x846ca68bU;
  x ^= x >> 16;
  return x;
}

// Two random bf16 values with exponent near 1 (sign, 7 random mantissa bits,
// exponent 126 or 127), packed.
__device__ __forceinline__ uint32_t rnd_bf16x2(uint32_t h) {
  const uint32_t lo = 0x3f00u | (h & 0x807fu) | ((h >> 7) & 0x80u);
  const uint32_t hi = 0x3f00u | ((h >> 16) & 0x807fu) | ((h >> 23) & 0x80u);
  return lo | (hi << 16);
}

__device__ __forceinline__ v4u rnd_frag(uint32_t seed) {
  return v4u{rnd_bf16x2(mix(seed)), rnd_bf16x2(mix(seed + 1)), rnd_bf16x2(mix(seed + 2)),
             rnd_bf16x2(mix(seed + 3))};
}

// New operand bits from old ones (x mixed with a shifted y), kept in the bf16
// pattern of rnd_bf16x2: three VALU operations per dword.
__device__ __forceinline__ v4u step(v4u x, v4u y) {
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = ((x[i] ^ (x[i] >> 3) ^ y[i]) & 0x80ff80ffu) | 0x3f003f00u;
  return x;
}

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_mfma_probe(int64_t iters, int mode, float* out, int64_t* clk) {
  const uint64_t c0 = __builtin_amdgcn_s_memtime();
  const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
  const uint32_t seed = (blockIdx.x * 256u + threadIdx.x) * 64u;
  v4u a[4], b[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (mode == 1) {
      a[i] = v4u{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u};
      b[i] = a[i];
    } else {
      a[i] = rnd_frag(seed + 8 * i);
      b[i] = rnd_frag(seed + 8 * i + 4 + 32);
    }
  }
  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};
  const bool refresh = mode == 2;
  for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a[i]),
                                                           __builtin_bit_cast(bf16x8_t, b[j]), acc[i][j], 0, 0, 0);
    if (refresh) {
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = step(a[i], b[(i + 1) & 3]);
    }
  }
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x;
        asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x) : "a"(acc[i][j][r]));
        s += x;
      }
  out[blockIdx.x * 256 + threadIdx.x] = s;
  if (threadIdx.x == 0) {
    const uint64_t c1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    clk[3 * blockIdx.x] = static_cast<int64_t>(c1 - c0);
    clk[3 * blockIdx.x + 1] = static_cast<int64_t>(r0);
    clk[3 * blockIdx.x + 2] = static_cast<int64_t>(r1);
  }
}

}  // namespace

// Launches `blocks` workgroups of 4 waves, each wave running `iters` rounds of
// 16 MFMAs (16 x 32 x 32 x 16 x 2 flops per round). out: blocks * 256 floats;
// clk: blocks * 3 int64 (per-workgroup s_memtime cycles, s_memrealtime start and
// end). Returns the HIP status of the launch.
extern "C" int sao_probe_mfma(int64_t blocks, int64_t iters, int mode, float* out, int64_t* clk,
                              hipStream_t stream) {
  if (blocks < 1 || blocks > (int64_t{1} << 20) || iters < 1 || mode < 0 || mode > 2 || !out || !clk)
    return static_cast<int>(hipErrorInvalidValue);
  hipLaunchKernelGGL(k_mfma_probe, dim3(static_cast<unsigned>(blocks)), dim3(256), 0, stream, iters, mode, out, clk);
  return static_cast<int>(hipGetLastError());
}

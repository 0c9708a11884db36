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
// mode 3: random operands read from LDS as the tile engine reads them: the
//         fragments of the next K step, one 16-byte read after each of the
//         first 8 MFMAs of a step, from a 2 x 64 KB ring of random bf16
// mode 4: mode 3 plus the engine's global -> LDS copies (16 global_load_lds_dwordx4
//         per wave per 4-step slab into the other stage, from an L2-resident 2 MB
//         buffer) and one copy wait and workgroup barrier per slab
// mode 5: mode 3 with both operands stored MN-major ([k][256 elements]) and read
//         through the transposing LDS read (ds_read_b64_tr_b16), two reads per
//         fragment, as the backward's dW product reads them
// mode 6: mode 5 plus the copies, copy wait and barrier of mode 4
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

__device__ __forceinline__ void pin() { __builtin_amdgcn_sched_barrier(0); }
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r / 2) % 8); }

struct Frags {
  v4u a[4];
  v4u b[4];
};

// Fragment idx of K step s (first-use order A0, B0 .. B3, A1 .. A3) from a
// 64 KB stage holding 256 A rows then 256 B rows of 8 16-byte chunks.
__device__ __forceinline__ void read_one(Frags& f, int idx, const v4u* l, int s, int wm, int wn, int lane) {
  const bool is_a = idx == 0 || idx > 4;
  const int i = idx == 0 ? 0 : (is_a ? idx - 4 : idx - 1);
  const int r32 = lane & 31;
  const int c = 2 * s + (lane >> 5);
  const int row0 = is_a ? wm * 128 : 256 + wn * 128;
  const v4u x = l[(row0 + r32) * 8 + swz(r32, c) + i * 32 * 8];
  if (is_a)
    f.a[i] = x;
  else
    f.b[i] = x;
}

typedef short v4i16_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16_t lds_v4i16_t;

// The same fragment from a stage holding an MN-major A slab (64 rows of K, 256
// elements each, 16-byte chunk c of row k at c ^ 4 (k & 3)) and then the B slab
// in the same form: within each 16 lanes, lane j names 4 elements of row
// k0 + (j >> 2) and receives column j of that 4 x 16 block; two reads give the
// 8 k values of the lane's half.
__device__ __forceinline__ void read_one_mn(Frags& f, int idx, const v4u* l, int s, int wm, int wn, int lane) {
  const bool is_a = idx == 0 || idx > 4;
  const int i = idx == 0 ? 0 : (is_a ? idx - 4 : idx - 1);
  const char* base = reinterpret_cast<const char*>(l) + (is_a ? 0 : 32768);
  const int j = lane & 15;
  const int k = 8 * (2 * s + (lane >> 5)) + (j >> 2);
  const int m = (is_a ? wm : wn) * 128 + 32 * i + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
  const int off = k * 512 + (((m >> 3) ^ (4 * (k & 3))) * 16) + (m & 7) * 2;
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(base + off));
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)(base + off + 4 * 512));
  const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
  const v4u x = v4u{a.x, a.y, b.x, b.y};
  if (is_a)
    f.a[i] = x;
  else
    f.b[i] = x;
}

__device__ __forceinline__ void dma16(const void* g, uint32_t off, uint32_t lds_base, uint32_t lds_off) {
  asm volatile("s_add_u32 m0, %2, %3\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(g), "s"(lds_base),
               "s"(lds_off)
               : "memory", "m0", "scc");
}

// Modes 3 and 4 (kCopies), 5 and 6 (kMn and kCopies): iters K steps of 16
// MFMAs each, in slabs of 4 steps.
template <bool kCopies, bool kMn>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_lds_probe(int64_t iters, const v4u* src, float* out, int64_t* clk) {
  __shared__ v4u lds[2][4096];
  const uint64_t c0 = __builtin_amdgcn_s_memtime();
  const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / 2, wn = wave % 2;
  const uint32_t seed = (blockIdx.x * 256u + tid) * 64u;
  for (int i = tid; i < 2 * 4096; i += 256) lds[i / 4096][i % 4096] = rnd_frag(seed + 4 * i);
  __syncthreads();
  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};
  Frags f0, f1;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f0.a[i] = rnd_frag(seed + 8 * i);
    f0.b[i] = rnd_frag(seed + 8 * i + 36);
  }
  f1 = f0;
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(&lds[0][0]));
  const uint32_t src_off = static_cast<uint32_t>(tid) * 16u;
  for (int64_t it = 0; it < iters / 4; ++it) {
    const int stage = static_cast<int>(it & 1);
    const v4u* l = lds[stage];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      Frags& cur = s % 2 == 0 ? f0 : f1;
      Frags& nxt = s % 2 == 0 ? f1 : f0;
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        acc[t / 4][t % 4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, cur.a[t / 4]),
                                                                    __builtin_bit_cast(bf16x8_t, cur.b[t % 4]),
                                                                    acc[t / 4][t % 4], 0, 0, 0);
        pin();
        if (t < 8) {
          if constexpr (kMn)
            read_one_mn(nxt, t, l, (s + 1) & 3, wm, wn, lane);
          else
            read_one(nxt, t, l, (s + 1) & 3, wm, wn, lane);
        }
        if constexpr (kCopies) {
          if ((s == 3 || s == 0) && (t & 1)) {
            // copy q of this wave: 1 KB of a 64 KB source window (32 windows in 2 MB)
            const int q = (s == 3 ? 0 : 8) + (t >> 1);
            const char* g = reinterpret_cast<const char*>(src) + (static_cast<int64_t>(it & 31) << 16) + q * 4096;
            dma16(g, src_off, lds0 + static_cast<uint32_t>((stage ^ 1) * 4096 * 16),
                  static_cast<uint32_t>((wave * 16 + q) * 1024));
          }
        }
        pin();
      }
      if constexpr (kCopies) {
        if (s == 2) {
          asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
          __builtin_amdgcn_s_barrier();
        }
      }
    }
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  float sum = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float x;
        asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x) : "a"(acc[i][j][r]));
        sum += x;
      }
  out[blockIdx.x * 256 + tid] = sum;
  if (tid == 0) {
    const uint64_t c1 = __builtin_amdgcn_s_memtime();
    const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
    clk[3 * blockIdx.x] = static_cast<int64_t>(c1 - c0);
    clk[3 * blockIdx.x + 1] = static_cast<int64_t>(r0);
    clk[3 * blockIdx.x + 2] = static_cast<int64_t>(r1);
  }
}

}  // namespace

// Launches `blocks` workgroups of 4 waves, each wave running `iters` rounds of
// 16 MFMAs (16 x 32 x 32 x 16 x 2 flops per round; modes 3 to 6 need iters a
// multiple of 4). src: for modes 4 and 6, a device buffer of at least 2 MB that the
// copies read (ignored otherwise). out: blocks * 256 floats; clk: blocks * 3
// int64 (per-workgroup s_memtime cycles, s_memrealtime start and end). Returns
// the HIP status of the launch.
extern "C" int sao_probe_mfma(int64_t blocks, int64_t iters, int mode, const void* src, float* out, int64_t* clk,
                              hipStream_t stream) {
  if (blocks < 1 || blocks > (int64_t{1} << 20) || iters < 1 || mode < 0 || mode > 6 || !out || !clk)
    return static_cast<int>(hipErrorInvalidValue);
  if (mode >= 3 && (iters % 4 != 0 || ((mode == 4 || mode == 6) && !src)))
    return static_cast<int>(hipErrorInvalidValue);
  const unsigned g = static_cast<unsigned>(blocks);
  if (mode <= 2)
    hipLaunchKernelGGL(k_mfma_probe, dim3(g), dim3(256), 0, stream, iters, mode, out, clk);
  else if (mode == 3)
    hipLaunchKernelGGL((k_lds_probe<false, false>), dim3(g), dim3(256), 0, stream, iters,
                       static_cast<const v4u*>(src), out, clk);
  else if (mode == 4)
    hipLaunchKernelGGL((k_lds_probe<true, false>), dim3(g), dim3(256), 0, stream, iters,
                       static_cast<const v4u*>(src), out, clk);
  else if (mode == 5)
    hipLaunchKernelGGL((k_lds_probe<false, true>), dim3(g), dim3(256), 0, stream, iters,
                       static_cast<const v4u*>(src), out, clk);
  else
    hipLaunchKernelGGL((k_lds_probe<true, true>), dim3(g), dim3(256), 0, stream, iters,
                       static_cast<const v4u*>(src), out, clk);
  return static_cast<int>(hipGetLastError());
}

// Block reductions, the loss-mask count and the token walk shared by the per-token
// kernels. Every reduction here runs in a fixed order, so results do not depend on
// scheduling.
#pragma once

#include "common.hpp"

namespace sao {

// Sum over a block of THREADS threads (a multiple of 64); every thread gets the
// result. `sh` holds THREADS / 64 elements.
template <int THREADS, typename T>
__device__ __forceinline__ T block_sum(T v, T* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  T r = sh[0];
#pragma unroll
  for (int w = 1; w < THREADS / 64; ++w) r += sh[w];
  return r;
}

// Per-block partial sums of the mask (grid-stride), then their total.
template <int THREADS>
__global__ __launch_bounds__(THREADS) void k_mask_count(const uint8_t* mask, int64_t T, int64_t* part) {
  __shared__ int64_t sh[THREADS / 64];
  int64_t c = 0;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * THREADS + threadIdx.x; t < T;
       t += static_cast<int64_t>(gridDim.x) * THREADS)
    c += mask[t] != 0 ? 1 : 0;
  c = block_sum<THREADS>(c, sh);
  if (threadIdx.x == 0) part[blockIdx.x] = c;
}

template <int THREADS>
__global__ __launch_bounds__(THREADS) void k_count_total(const int64_t* part, int nblk, int64_t* total) {
  __shared__ int64_t sh[THREADS / 64];
  int64_t c = 0;
  for (int i = threadIdx.x; i < nblk; i += THREADS) c += part[i];
  c = block_sum<THREADS>(c, sh);
  if (threadIdx.x == 0) *total = c;
}

// Token walk of the per-token kernels. Each wave takes chunks of 512 consecutive
// tokens (grid-stride over chunks); lane l handles tokens 4l .. 4l+3 and
// 256 + 4l .. 256 + 4l+3 of a chunk, so every load and store instruction of a
// whole chunk covers one contiguous span. quad(t) handles tokens t .. t+3 with
// 16-byte vector access (whole chunks, when vec_ok); one(t) handles a single
// token (the ragged tail, or every token when the bases do not allow vectors).
constexpr int kWalkChunk = 512;

template <int THREADS, class Quad, class One>
__device__ __forceinline__ void walk_tokens(int64_t T, bool vec_ok, Quad&& quad, One&& one) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t waves = static_cast<int64_t>(gridDim.x) * (THREADS / 64);
  for (int64_t w0 = (static_cast<int64_t>(blockIdx.x) * (THREADS / 64) + wave) * kWalkChunk; w0 < T;
       w0 += waves * kWalkChunk) {
    if (vec_ok && w0 + kWalkChunk <= T) {
#pragma unroll
      for (int half = 0; half < 2; ++half) quad(w0 + half * (kWalkChunk / 2) + 4 * lane);
    } else {
      for (int j = 0; j < 8; ++j) {
        const int64_t t = w0 + (j < 4 ? 4 * lane + j : kWalkChunk / 2 + 4 * lane + (j - 4));
        if (t < T) one(t);
      }
    }
  }
}

}  // namespace sao

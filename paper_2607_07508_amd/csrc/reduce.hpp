// Block reductions and the loss-mask count shared by the loss and value kernels.
// Every reduction here runs in a fixed order, so results do not depend on
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

}  // namespace sao

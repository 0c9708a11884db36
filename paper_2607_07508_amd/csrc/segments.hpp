// Validation of the packed trajectory segments shared by the advantage kernels.
#pragma once

#include "common.hpp"
#include "../../include/sao.h"

namespace sao {

// One block: cu_seqlens must rise from 0 to T without decreasing. Sets *bad (0/1),
// zeroes *n_tokens, and flags the status word.
template <int THREADS>
__global__ __launch_bounds__(THREADS) void k_check_segments(const int32_t* cu, int32_t B, int64_t T, int32_t* bad,
                                                            int64_t* n_tokens, int32_t* status) {
  __shared__ int32_t s_bad;
  if (threadIdx.x == 0) s_bad = (cu[0] != 0 || static_cast<int64_t>(cu[B]) != T) ? 1 : 0;
  __syncthreads();
  for (int32_t i = threadIdx.x; i < B; i += THREADS)
    if (cu[i + 1] < cu[i]) atomicOr(&s_bad, 1);
  __syncthreads();
  if (threadIdx.x == 0) {
    *bad = s_bad;
    if (n_tokens) *n_tokens = 0;
    if (s_bad && status) atomicOr(status, SAO_STATUS_SEGMENTS);
  }
}

// Malformed segments: block blockIdx.x of B writes NaN advantages (and NaN
// returns and 0 to `last`, when given) over an even slice of [0, T), and adds
// that slice's mask count to *n_tokens.
template <int THREADS>
__device__ __forceinline__ void malformed_slice(const uint8_t* mask, int32_t B, int64_t T, float* adv, float* ret,
                                                uint8_t* last, int64_t* n_tokens) {
  const int64_t b = blockIdx.x;
  const int64_t lo = T * b / B, hi = T * (b + 1) / B;
  int64_t cnt = 0;
  for (int64_t t = lo + threadIdx.x; t < hi; t += THREADS) {
    adv[t] = __builtin_nanf("");
    if (ret) ret[t] = __builtin_nanf("");
    if (last) last[t] = 0;
    cnt += mask[t] != 0 ? 1 : 0;
  }
  cnt = wave_sum(cnt);
  if ((threadIdx.x & 63) == 0 && n_tokens && cnt)
    atomicAdd(reinterpret_cast<unsigned long long*>(n_tokens), static_cast<unsigned long long>(cnt));
}

}  // namespace sao

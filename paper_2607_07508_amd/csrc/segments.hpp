// Validation of the packed trajectory segments and the loss-mask count shared by
// the advantage kernels.
#pragma once

#include "common.hpp"
#include "../../include/sao.h"

namespace sao {

// One block: cu_seqlens must rise from 0 to T without decreasing. Sets *bad (0/1),
// zeroes the kSlots count slots, and flags the status word.
template <int THREADS, int kSlots>
__global__ __launch_bounds__(THREADS) void k_check_segments(const int32_t* cu, int32_t B, int64_t T, int32_t* bad,
                                                            int64_t* slots, int32_t* status) {
  __shared__ int32_t s_bad;
  if (threadIdx.x == 0) s_bad = (cu[0] != 0 || static_cast<int64_t>(cu[B]) != T) ? 1 : 0;
  for (int i = threadIdx.x; i < kSlots; i += THREADS) slots[i] = 0;
  __syncthreads();
  for (int32_t i = threadIdx.x; i < B; i += THREADS)
    if (cu[i + 1] < cu[i]) atomicOr(&s_bad, 1);
  __syncthreads();
  if (threadIdx.x == 0) {
    *bad = s_bad;
    if (s_bad && status) atomicOr(status, SAO_STATUS_SEGMENTS);
  }
}

// Adds a workgroup's loss-mask count to its slot. Many workgroups adding to one
// address serialise at the cache; spread over the slots they do not.
template <int kSlots>
__device__ __forceinline__ void add_count(int64_t* slots, int64_t cnt) {
  if (cnt) atomicAdd(reinterpret_cast<unsigned long long*>(slots + blockIdx.x % kSlots), static_cast<unsigned long long>(cnt));
}

// *n_tokens = the sum of the kSlots slots (one wave).
template <int kSlots>
__global__ __launch_bounds__(64) void k_slots_total(const int64_t* slots, int64_t* n_tokens) {
  static_assert(kSlots == 64, "one slot per lane");
  const int64_t v = wave_sum(slots[threadIdx.x]);
  if (threadIdx.x == 0) *n_tokens = v;
}

// Malformed segments: block blockIdx.x of B writes NaN advantages (and NaN
// returns and 0 to `last`, when given) over an even slice of [0, T), and adds
// that slice's mask count to its count slot.
template <int THREADS, int kSlots>
__device__ __forceinline__ void malformed_slice(const uint8_t* mask, int32_t B, int64_t T, float* adv, float* ret,
                                                uint8_t* last, int64_t* slots) {
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
  if ((threadIdx.x & 63) == 0) add_count<kSlots>(slots, cnt);
}

}  // namespace sao

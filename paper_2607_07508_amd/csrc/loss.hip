// Direct double-sided importance sampling and the token-level mean (Sec. 3.1, Eq. 1-3).
//
// One pass over the tokens: rho = exp(logp - logp_rollout) in float64, the strict
// band flag, g = d loss / d logp, and per-block partial sums (loss terms in
// float64, counts in int64) reduced in a fixed order by a one-block final kernel,
// so results do not depend on scheduling.
#include "common.hpp"
#include "launch.hpp"
#include "layout.hpp"
#include "reduce.hpp"
#include "../../include/sao.h"

namespace sao {

// Per-thread running sums of one call.
struct LossAcc {
  double sL = 0.0, sS = 0.0;
  int64_t c[5] = {0, 0, 0, 0, 0};
};

// One loss-mask token: rho in float64 (Eq. 2), the strict band (Eq. 3), and
// the token's share of the mean (Eq. 1). Returns the flag; writes g.
__device__ __forceinline__ uint8_t loss_token(bool active, float lpf, float lrof, float advf, double lo, double hi,
                                              int64_t N, double invN, LossAcc& acc, float& g) {
  g = 0.0f;
  if (!active) return SAO_FLAG_MASKED;
  ++acc.c[0];
  const double lp = lpf;
  const double rho = exp(lp - static_cast<double>(lrof));
  uint8_t f;
  if (__builtin_isnan(rho))
    f = SAO_FLAG_NONFINITE;
  else if (rho <= lo)
    f = SAO_FLAG_LOW;
  else if (rho >= hi)
    f = SAO_FLAG_HIGH;
  else
    f = SAO_FLAG_USED;  // 1 - eps_l < rho < 1 + eps_h
  ++acc.c[f];
  if (f == SAO_FLAG_USED && N > 0) {
    const double w = rho * static_cast<double>(advf);
    acc.sL = fma(w, lp, acc.sL);
    acc.sS += w;
    g = static_cast<float>(-w * invN);
  }
  return f;
}

// Each thread takes groups of kLossPerThread consecutive tokens (grid-stride
// over groups); whole groups use 16-byte vector accesses when the bases allow.
__global__ __launch_bounds__(kLossThreads) void k_loss(const float* logp, const float* lro, const float* adv,
                                                       const uint8_t* mask, int64_t T, float eps_low,
                                                       float eps_high, const int64_t* n_ptr, double* part_f,
                                                       int64_t* part_i, float* g, uint8_t* flags, bool vec_ok) {
  static_assert(kLossPerThread == 8, "vector path handles 8 tokens per group");
  __shared__ double shd[kLossThreads / 64];
  __shared__ int64_t shi[kLossThreads / 64];
  const int64_t N = *n_ptr;
  const double lo = 1.0 - static_cast<double>(eps_low);
  const double hi = 1.0 + static_cast<double>(eps_high);
  const double invN = N > 0 ? 1.0 / static_cast<double>(N) : 0.0;
  LossAcc acc;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kLossThreads * kLossPerThread;
  for (int64_t t0 = (static_cast<int64_t>(blockIdx.x) * kLossThreads + threadIdx.x) * kLossPerThread; t0 < T;
       t0 += stride) {
    if (vec_ok && t0 + kLossPerThread <= T) {
      const f32x4_t* pl = reinterpret_cast<const f32x4_t*>(logp + t0);
      const f32x4_t* pr = reinterpret_cast<const f32x4_t*>(lro + t0);
      const f32x4_t* pa = reinterpret_cast<const f32x4_t*>(adv + t0);
      const f32x4_t l0 = pl[0], l1 = pl[1], r0 = pr[0], r1 = pr[1], a0 = pa[0], a1 = pa[1];
      const uint2 m8 = *reinterpret_cast<const uint2*>(mask + t0);
      float gg[8];
      uint32_t fl[2] = {0u, 0u};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t mw = j < 4 ? m8.x : m8.y;
        const bool act = ((mw >> (8 * (j & 3))) & 0xffu) != 0;
        const float lpv = j < 4 ? l0[j & 3] : l1[j & 3];
        const float lrv = j < 4 ? r0[j & 3] : r1[j & 3];
        const float adv_ = j < 4 ? a0[j & 3] : a1[j & 3];
        const uint8_t f = loss_token(act, lpv, lrv, adv_, lo, hi, N, invN, acc, gg[j]);
        fl[j >> 2] |= static_cast<uint32_t>(f) << (8 * (j & 3));
      }
      f32x4_t* pg = reinterpret_cast<f32x4_t*>(g + t0);
      pg[0] = f32x4_t{gg[0], gg[1], gg[2], gg[3]};
      pg[1] = f32x4_t{gg[4], gg[5], gg[6], gg[7]};
      *reinterpret_cast<uint2*>(flags + t0) = uint2{fl[0], fl[1]};
    } else {
      for (int j = 0; j < kLossPerThread; ++j) {
        const int64_t t = t0 + j;
        if (t >= T) break;
        const bool act = mask[t] != 0;
        float gt;
        flags[t] = loss_token(act, act ? logp[t] : 0.0f, act ? lro[t] : 0.0f, act ? adv[t] : 0.0f, lo, hi, N,
                              invN, acc, gt);
        g[t] = gt;
      }
    }
  }
  const double sL = block_sum<kLossThreads>(acc.sL, shd);
  const double sS = block_sum<kLossThreads>(acc.sS, shd);
  int64_t tot[5];
#pragma unroll
  for (int i = 0; i < 5; ++i) tot[i] = block_sum<kLossThreads>(acc.c[i], shi);
  if (threadIdx.x == 0) {
    part_f[2 * blockIdx.x] = sL;
    part_f[2 * blockIdx.x + 1] = sS;
#pragma unroll
    for (int i = 0; i < 5; ++i) part_i[5 * blockIdx.x + i] = tot[i];
  }
}

__global__ __launch_bounds__(kLossThreads) void k_loss_final(const double* part_f, const int64_t* part_i,
                                                             int nblk, const int64_t* n_ptr, double* loss,
                                                             int64_t* counts) {
  __shared__ double shd[kLossThreads / 64];
  __shared__ int64_t shi[kLossThreads / 64];
  double sL = 0.0, sS = 0.0;
  int64_t c[5] = {0, 0, 0, 0, 0};
  for (int i = threadIdx.x; i < nblk; i += kLossThreads) {
    sL += part_f[2 * i];
    sS += part_f[2 * i + 1];
#pragma unroll
    for (int k = 0; k < 5; ++k) c[k] += part_i[5 * i + k];
  }
  sL = block_sum<kLossThreads>(sL, shd);
  sS = block_sum<kLossThreads>(sS, shd);
  int64_t tot[5];
#pragma unroll
  for (int k = 0; k < 5; ++k) tot[k] = block_sum<kLossThreads>(c[k], shi);
  if (threadIdx.x == 0) {
    const int64_t N = *n_ptr;
    if (N > 0) {
      loss[0] += -sL / static_cast<double>(N);
      loss[1] += -sS / static_cast<double>(N);
    }
#pragma unroll
    for (int k = 0; k < 5; ++k) counts[k] += tot[k];
  }
}

hipError_t launch_loss(const float* logp, const float* logp_rollout, const float* adv, const uint8_t* mask,
                       int64_t T, float eps_low, float eps_high, const int64_t* n_tokens, double* loss,
                       float* g, uint8_t* flags, int64_t* counts, void* ws, hipStream_t st) {
  const LossLayout L = loss_layout(T);
  char* w8 = static_cast<char*>(ws);
  double* part_f = reinterpret_cast<double*>(w8 + L.part_f);
  int64_t* part_i = reinterpret_cast<int64_t*>(w8 + L.part_i);
  const int nblk = static_cast<int>(L.blocks);
  const int64_t* n_ptr = n_tokens;
  if (!n_ptr) {
    int64_t* total = reinterpret_cast<int64_t*>(w8 + L.n_count);
    hipLaunchKernelGGL(k_mask_count<kLossThreads>, dim3(nblk), dim3(kLossThreads), 0, st, mask, T, part_i);
    hipLaunchKernelGGL(k_count_total<kLossThreads>, dim3(1), dim3(kLossThreads), 0, st, part_i, nblk, total);
    n_ptr = total;
  }
  const uintptr_t f = reinterpret_cast<uintptr_t>(logp) | reinterpret_cast<uintptr_t>(logp_rollout) |
                      reinterpret_cast<uintptr_t>(adv) | reinterpret_cast<uintptr_t>(g);
  const bool vec_ok = (f & 15u) == 0 && ((reinterpret_cast<uintptr_t>(mask) | reinterpret_cast<uintptr_t>(flags)) & 7u) == 0;
  hipLaunchKernelGGL(k_loss, dim3(nblk), dim3(kLossThreads), 0, st, logp, logp_rollout, adv, mask, T,
                     eps_low, eps_high, n_ptr, part_f, part_i, g, flags, vec_ok);
  hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(kLossThreads), 0, st, part_f, part_i, nblk, n_ptr, loss,
                     counts);
  return hipGetLastError();
}

}  // namespace sao

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

__global__ __launch_bounds__(kLossThreads) void k_loss(const float* logp, const float* lro, const float* adv,
                                                       const uint8_t* mask, int64_t T, float eps_low,
                                                       float eps_high, const int64_t* n_ptr, double* part_f,
                                                       int64_t* part_i, float* g, uint8_t* flags) {
  __shared__ double shd[kLossThreads / 64];
  __shared__ int64_t shi[kLossThreads / 64];
  const int64_t N = *n_ptr;
  const double lo = 1.0 - static_cast<double>(eps_low);
  const double hi = 1.0 + static_cast<double>(eps_high);
  const double invN = N > 0 ? 1.0 / static_cast<double>(N) : 0.0;
  double sL = 0.0, sS = 0.0;
  int64_t c[5] = {0, 0, 0, 0, 0};
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * kLossThreads + threadIdx.x; t < T;
       t += static_cast<int64_t>(gridDim.x) * kLossThreads) {
    if (mask[t] == 0) {
      flags[t] = SAO_FLAG_MASKED;
      g[t] = 0.0f;
      continue;
    }
    ++c[0];
    const double lp = logp[t];
    const double rho = exp(lp - static_cast<double>(lro[t]));  // Eq. (2)
    uint8_t f;
    if (__builtin_isnan(rho))
      f = SAO_FLAG_NONFINITE;
    else if (rho <= lo)
      f = SAO_FLAG_LOW;
    else if (rho >= hi)
      f = SAO_FLAG_HIGH;
    else
      f = SAO_FLAG_USED;                                       // 1 - eps_l < rho < 1 + eps_h, Eq. (3)
    flags[t] = f;
    ++c[f];
    float gt = 0.0f;
    if (f == SAO_FLAG_USED && N > 0) {
      const double w = rho * static_cast<double>(adv[t]);
      sL = fma(w, lp, sL);
      sS += w;
      gt = static_cast<float>(-w * invN);
    }
    g[t] = gt;
  }
  sL = block_sum<kLossThreads>(sL, shd);
  sS = block_sum<kLossThreads>(sS, shd);
  int64_t tot[5];
#pragma unroll
  for (int i = 0; i < 5; ++i) tot[i] = block_sum<kLossThreads>(c[i], shi);
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
  hipLaunchKernelGGL(k_loss, dim3(nblk), dim3(kLossThreads), 0, st, logp, logp_rollout, adv, mask, T,
                     eps_low, eps_high, n_ptr, part_f, part_i, g, flags);
  hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(kLossThreads), 0, st, part_f, part_i, nblk, n_ptr, loss,
                     counts);
  return hipGetLastError();
}

}  // namespace sao

// Direct double-sided importance sampling and the token-level mean (Sec. 3.1, Eq. 1-3).
//
// One pass over the tokens: the strict band flag of rho = exp(logp - logp_rollout),
// decided exactly as in float64, g = d loss / d logp, and per-block partial sums
// (loss terms in float64, counts in int64) reduced in a fixed order by a one-block
// final kernel, so results do not depend on scheduling.
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

// The band edges of Eq. (3) in ratio and in log-ratio space.
struct Band {
  double lo, hi, ln_lo, ln_hi;
};

// Whether d lies within a margin of a band edge in log space. fp64 exp is
// faithful to about one ulp, so outside 1e-12 (relative) comparing
// d = logp - logp_rollout with ln(1 -+ eps) decides exactly as comparing
// exp(d) with 1 -+ eps; inside, the ratio itself is compared.
__device__ __forceinline__ bool near_edge(double d, double edge) {
  return fabs(d - edge) <= 1e-12 * fmax(1.0, fabs(edge));
}

// One loss-mask token: the strict band of Eq. (3) on rho = exp(logp - logp_rollout)
// (Eq. 2), decided as in float64, and the token's share of the mean (Eq. 1), whose
// weight rho is evaluated in float32. Returns the flag; writes g.
__device__ __forceinline__ uint8_t loss_token(bool active, float lpf, float lrof, float advf, const Band& bd,
                                              int64_t N, double invN, LossAcc& acc, float& g) {
  g = 0.0f;
  if (!active) return SAO_FLAG_MASKED;
  ++acc.c[0];
  const double lp = lpf;
  const double d = lp - static_cast<double>(lrof);
  uint8_t f;
  if (__builtin_isnan(d)) {
    f = SAO_FLAG_NONFINITE;
  } else {
    bool low;
    if (bd.lo > 0.0)
      low = near_edge(d, bd.ln_lo) ? exp(d) <= bd.lo : d < bd.ln_lo;
    else  // rho > 0 unless exp underflows
      low = d < -700.0 ? exp(d) <= bd.lo : false;
    const bool high = near_edge(d, bd.ln_hi) ? exp(d) >= bd.hi : d > bd.ln_hi;
    f = low ? SAO_FLAG_LOW : (high ? SAO_FLAG_HIGH : SAO_FLAG_USED);  // 1 - eps_l < rho < 1 + eps_h
  }
  ++acc.c[f];
  if (f == SAO_FLAG_USED && N > 0) {
    const double rho = fast_exp2(static_cast<float>(d) * kLog2e);
    const double w = rho * static_cast<double>(advf);
    acc.sL = fma(w, lp, acc.sL);
    acc.sS += w;
    g = static_cast<float>(-w * invN);
  }
  return f;
}

// Each wave takes chunks of 512 consecutive tokens (grid-stride over chunks);
// lane l handles tokens 4l .. 4l+3 and 256 + 4l .. 256 + 4l+3 of a chunk, so every
// load and store instruction of a whole chunk covers one contiguous span (when
// the bases allow vector access).
__global__ __launch_bounds__(kLossThreads) void k_loss(const float* logp, const float* lro, const float* adv,
                                                       const uint8_t* mask, int64_t T, float eps_low,
                                                       float eps_high, const int64_t* n_ptr, double* part_f,
                                                       int64_t* part_i, float* g, uint8_t* flags, bool vec_ok) {
  static_assert(kLossPerThread == 8, "a wave chunk is 64 lanes x 8 tokens");
  constexpr int kChunk = 64 * kLossPerThread;
  __shared__ double shd[kLossThreads / 64];
  __shared__ int64_t shi[kLossThreads / 64];
  const int64_t N = *n_ptr;
  Band bd;
  bd.lo = 1.0 - static_cast<double>(eps_low);
  bd.hi = 1.0 + static_cast<double>(eps_high);
  bd.ln_lo = bd.lo > 0.0 ? log(bd.lo) : 0.0;
  bd.ln_hi = log(bd.hi);
  const double invN = N > 0 ? 1.0 / static_cast<double>(N) : 0.0;
  LossAcc acc;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t waves = static_cast<int64_t>(gridDim.x) * (kLossThreads / 64);
  for (int64_t w0 = (static_cast<int64_t>(blockIdx.x) * (kLossThreads / 64) + wave) * kChunk; w0 < T;
       w0 += waves * kChunk) {
    if (vec_ok && w0 + kChunk <= T) {
#pragma unroll
      for (int half = 0; half < 2; ++half) {
        const int64_t t = w0 + half * (kChunk / 2) + 4 * lane;
        const f32x4_t l4 = *reinterpret_cast<const f32x4_t*>(logp + t);
        const f32x4_t r4 = *reinterpret_cast<const f32x4_t*>(lro + t);
        const f32x4_t a4 = *reinterpret_cast<const f32x4_t*>(adv + t);
        const uint32_t m4 = *reinterpret_cast<const uint32_t*>(mask + t);
        float gg[4];
        uint32_t fl = 0u;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bool act = ((m4 >> (8 * j)) & 0xffu) != 0;
          fl |= static_cast<uint32_t>(loss_token(act, l4[j], r4[j], a4[j], bd, N, invN, acc, gg[j])) << (8 * j);
        }
        *reinterpret_cast<f32x4_t*>(g + t) = f32x4_t{gg[0], gg[1], gg[2], gg[3]};
        *reinterpret_cast<uint32_t*>(flags + t) = fl;
      }
    } else {
      for (int j = 0; j < kLossPerThread; ++j) {
        const int64_t t = w0 + (j < 4 ? 4 * lane + j : kChunk / 2 + 4 * lane + (j - 4));
        if (t >= T) continue;
        const bool act = mask[t] != 0;
        float gt;
        flags[t] = loss_token(act, act ? logp[t] : 0.0f, act ? lro[t] : 0.0f, act ? adv[t] : 0.0f, bd, N,
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
  const bool vec_ok = (f & 15u) == 0 && ((reinterpret_cast<uintptr_t>(mask) | reinterpret_cast<uintptr_t>(flags)) & 3u) == 0;
  hipLaunchKernelGGL(k_loss, dim3(nblk), dim3(kLossThreads), 0, st, logp, logp_rollout, adv, mask, T,
                     eps_low, eps_high, n_ptr, part_f, part_i, g, flags, vec_ok);
  hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(kLossThreads), 0, st, part_f, part_i, nblk, n_ptr, loss,
                     counts);
  return hipGetLastError();
}

}  // namespace sao

// Direct double-sided importance sampling and the token-level mean (Sec. 3.1, Eq. 1-3),
// and the clipped surrogate it is compared with (Sec. 2; decoupled form of Sec. 3.1).
//
// One pass over the tokens: the clip flag of the ratio, decided exactly as in
// float64, g = d loss / d logp, and per-block partial sums (loss terms in float64,
// counts in int64) reduced in a fixed order by a one-block final kernel, so
// results do not depend on scheduling.
#include <mutex>

#include "common.hpp"
#include "launch.hpp"
#include "layout.hpp"
#include "reduce.hpp"
#include "../../include/sao.h"

namespace sao {

static_assert(64 * kLossPerThread == kWalkChunk, "one wave chunk is 64 lanes x 8 tokens");

// Per-thread running sums of one call.
struct LossAcc {
  double sL = 0.0, sS = 0.0;
  int64_t c[5] = {0, 0, 0, 0, 0};
};

// Whether d lies within a margin of a band edge in log space. fp64 exp is
// faithful to about one ulp, so outside 1e-12 (relative) comparing
// d = log r with ln(1 -+ eps) decides exactly as comparing exp(d) with
// 1 -+ eps; inside, the ratio itself is compared.
__device__ __forceinline__ bool near_edge(double d, double edge) {
  return fabs(d - edge) <= 1e-12 * fmax(1.0, fabs(edge));
}

// The clip edges 1 - eps_low and 1 + eps_high, in ratio and in log-ratio space,
// and comparisons of a ratio r = exp(d) with them, decided as in float64.
struct Band {
  double lo, hi, ln_lo, ln_hi;

  __device__ Band(float eps_low, float eps_high) {
    lo = 1.0 - static_cast<double>(eps_low);
    hi = 1.0 + static_cast<double>(eps_high);
    ln_lo = lo > 0.0 ? log(lo) : 0.0;
    ln_hi = log(hi);
  }
  // r <= max(lo, 0), the lower edge of the DIS band. A ratio is never negative,
  // so with eps_low >= 1 only r = 0 (log pi = -inf, or exp underflow) falls below
  // the band; it is clipped low like a ratio at the edge.
  __device__ bool le_lo(double d) const {
    if (lo > 0.0) return near_edge(d, ln_lo) ? exp(d) <= lo : d < ln_lo;
    return d < -700.0 ? exp(d) <= 0.0 : false;  // r > 0 unless exp underflows
  }
  __device__ bool lt_lo(double d) const {  // r < lo
    if (lo > 0.0) return near_edge(d, ln_lo) ? exp(d) < lo : d < ln_lo;
    return false;
  }
  __device__ bool ge_hi(double d) const { return near_edge(d, ln_hi) ? exp(d) >= hi : d > ln_hi; }
  __device__ bool gt_hi(double d) const { return near_edge(d, ln_hi) ? exp(d) > hi : d > ln_hi; }
};

// One loss-mask token of the DIS objective: the strict band of Eq. (3) on
// rho = exp(logp - logp_rollout) (Eq. 2), decided as in float64, and the token's
// share of the mean (Eq. 1), whose weight rho is evaluated in float32. Returns
// the flag; writes g.
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
    const bool low = bd.le_lo(d), high = bd.ge_hi(d);
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

// One loss-mask token of the clipped surrogate of Sec. 2: r = exp(logp - logp_old),
// clipped exactly when A > 0 and r > 1 + eps_high or A < 0 and r < 1 - eps_low, and
// with kWeighted the decoupled weight w = exp(logp_old - logp_behav) of Sec. 3.1 (a
// constant). The term w min(r A, clip(r) A) goes into sL; g = -w r A / N on unclipped
// tokens. Everything is float64, so ratios far outside the band stay finite.
template <bool kWeighted>
__device__ __forceinline__ uint8_t ppo_token(bool active, float lpf, float loldf, float lbf, float advf,
                                             const Band& bd, int64_t N, double invN, LossAcc& acc, float& g) {
  g = 0.0f;
  if (!active) return SAO_FLAG_MASKED;
  ++acc.c[0];
  const double lold = loldf;
  const double d = static_cast<double>(lpf) - lold;
  const double e = kWeighted ? lold - static_cast<double>(lbf) : 0.0;
  const double A = advf;
  uint8_t f;
  if (__builtin_isnan(d) || __builtin_isnan(e))
    f = SAO_FLAG_NONFINITE;
  else if (A > 0.0 && bd.gt_hi(d))
    f = SAO_FLAG_HIGH;
  else if (A < 0.0 && bd.lt_lo(d))
    f = SAO_FLAG_LOW;
  else
    f = SAO_FLAG_USED;
  ++acc.c[f];
  // Both exponentials are evaluated on every lane and the results selected, so
  // the wave does not branch on the flag.
  const double w = kWeighted ? exp(e) : 1.0;
  const double rd = exp(d);
  const double r = f == SAO_FLAG_USED ? rd : (f == SAO_FLAG_HIGH ? bd.hi : bd.lo);
  const double term = w * (r * A);
  const bool counted = f != SAO_FLAG_NONFINITE && N > 0;
  acc.sL += counted ? term : 0.0;
  if (counted && f == SAO_FLAG_USED) g = static_cast<float>(-term * invN);
  return f;
}

// The block's partial sums: part_f gets sL and sS, part_i the five counts.
__device__ __forceinline__ void store_partials(const LossAcc& acc, double* part_f, int64_t* part_i) {
  __shared__ double shd[kLossThreads / 64];
  __shared__ int64_t shi[kLossThreads / 64];
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

__global__ __launch_bounds__(kLossThreads) void k_loss(const float* logp, const float* lro, const float* adv,
                                                       const uint8_t* mask, int64_t T, float eps_low,
                                                       float eps_high, const int64_t* n_ptr, double* part_f,
                                                       int64_t* part_i, float* g, uint8_t* flags, bool vec_ok) {
  const int64_t N = *n_ptr;
  const Band bd(eps_low, eps_high);
  const double invN = N > 0 ? 1.0 / static_cast<double>(N) : 0.0;
  LossAcc acc;
  walk_tokens<kLossThreads>(
      T, vec_ok,
      [&](int64_t t) {
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
      },
      [&](int64_t t) {
        const bool act = mask[t] != 0;
        float gt;
        flags[t] = loss_token(act, act ? logp[t] : 0.0f, act ? lro[t] : 0.0f, act ? adv[t] : 0.0f, bd, N, invN,
                              acc, gt);
        g[t] = gt;
      });
  store_partials(acc, part_f, part_i);
}

template <bool kWeighted>
__global__ __launch_bounds__(kLossThreads) void k_ppo(const float* logp, const float* lold, const float* lb,
                                                      const float* adv, const uint8_t* mask, int64_t T,
                                                      float eps_low, float eps_high, const int64_t* n_ptr,
                                                      double* part_f, int64_t* part_i, float* g, uint8_t* flags,
                                                      bool vec_ok) {
  const int64_t N = *n_ptr;
  const Band bd(eps_low, eps_high);
  const double invN = N > 0 ? 1.0 / static_cast<double>(N) : 0.0;
  LossAcc acc;
  walk_tokens<kLossThreads>(
      T, vec_ok,
      [&](int64_t t) {
        const f32x4_t l4 = *reinterpret_cast<const f32x4_t*>(logp + t);
        const f32x4_t o4 = *reinterpret_cast<const f32x4_t*>(lold + t);
        const f32x4_t b4 = kWeighted ? *reinterpret_cast<const f32x4_t*>(lb + t) : f32x4_t{0.f, 0.f, 0.f, 0.f};
        const f32x4_t a4 = *reinterpret_cast<const f32x4_t*>(adv + t);
        const uint32_t m4 = *reinterpret_cast<const uint32_t*>(mask + t);
        float gg[4];
        uint32_t fl = 0u;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const bool act = ((m4 >> (8 * j)) & 0xffu) != 0;
          fl |= static_cast<uint32_t>(ppo_token<kWeighted>(act, l4[j], o4[j], b4[j], a4[j], bd, N, invN, acc, gg[j]))
                << (8 * j);
        }
        *reinterpret_cast<f32x4_t*>(g + t) = f32x4_t{gg[0], gg[1], gg[2], gg[3]};
        *reinterpret_cast<uint32_t*>(flags + t) = fl;
      },
      [&](int64_t t) {
        const bool act = mask[t] != 0;
        float gt;
        flags[t] = ppo_token<kWeighted>(act, act ? logp[t] : 0.0f, act ? lold[t] : 0.0f,
                                        (kWeighted && act) ? lb[t] : 0.0f, act ? adv[t] : 0.0f, bd, N, invN,
                                        acc, gt);
        g[t] = gt;
      });
  store_partials(acc, part_f, part_i);
}

// Sums the block partials in a fixed order; adds -sL/N (and, when n_loss == 2,
// -sS/N) to loss and the counts to counts.
__global__ __launch_bounds__(kLossThreads) void k_loss_final(const double* part_f, const int64_t* part_i,
                                                             int nblk, const int64_t* n_ptr, int n_loss,
                                                             double* loss, int64_t* counts) {
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
      if (n_loss > 1) loss[1] += -sS / static_cast<double>(N);
    }
#pragma unroll
    for (int k = 0; k < 5; ++k) counts[k] += tot[k];
  }
}

namespace {

// N from the caller, or the mask count of this call computed into the workspace.
const int64_t* token_count(const int64_t* n_tokens, const uint8_t* mask, int64_t T, const LossLayout& L,
                           char* w8, hipStream_t st) {
  if (n_tokens) return n_tokens;
  int64_t* part_i = reinterpret_cast<int64_t*>(w8 + L.part_i);
  int64_t* total = reinterpret_cast<int64_t*>(w8 + L.n_count);
  const int nblk = static_cast<int>(L.blocks);
  hipLaunchKernelGGL(k_mask_count<kLossThreads>, dim3(nblk), dim3(kLossThreads), 0, st, mask, T, part_i);
  hipLaunchKernelGGL(k_count_total<kLossThreads>, dim3(1), dim3(kLossThreads), 0, st, part_i, nblk, total);
  return total;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

}  // namespace

int launch_loss(const float* logp, const float* logp_rollout, const float* adv, const uint8_t* mask,
                       int64_t T, float eps_low, float eps_high, const int64_t* n_tokens, double* loss,
                       float* g, uint8_t* flags, int64_t* counts, void* ws, hipStream_t st) {
  const LossLayout L = loss_layout(T);
  char* w8 = static_cast<char*>(ws);
  double* part_f = reinterpret_cast<double*>(w8 + L.part_f);
  int64_t* part_i = reinterpret_cast<int64_t*>(w8 + L.part_i);
  const int nblk = static_cast<int>(L.blocks);
  const int64_t* n_ptr = token_count(n_tokens, mask, T, L, w8, st);
  const bool vec_ok = aligned(logp, 16) && aligned(logp_rollout, 16) && aligned(adv, 16) && aligned(g, 16) &&
                      aligned(mask, 4) && aligned(flags, 4);
  hipLaunchKernelGGL(k_loss, dim3(nblk), dim3(kLossThreads), 0, st, logp, logp_rollout, adv, mask, T,
                     eps_low, eps_high, n_ptr, part_f, part_i, g, flags, vec_ok);
  hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(kLossThreads), 0, st, part_f, part_i, nblk, n_ptr, 2, loss,
                     counts);
  return hipGetLastError();
}

// ------------------------------------------------------------------------- //
// sao_clipped_loss_noalloc: the same kernels with their workspace in a static
// device array instead of the caller's buffer, for callers that cannot allocate.
// ------------------------------------------------------------------------- //

// kLossScratchBytes: the loss layout at its largest. One copy per device (each GPU holds its own, at its own address, until the
// process ends). Host code never uses this name as an address: on the host it is
// only a handle for hipGetSymbolAddress.
static __device__ __align__(256) unsigned char scratch[kLossScratchBytes];

namespace {

constexpr int kMaxDevices = 64;

struct ScratchSlot {
  std::once_flag once;
  void* ptr = nullptr;
  hipError_t err = hipSuccess;
};
ScratchSlot g_scratch[kMaxDevices];

}  // namespace

int launch_loss_noalloc(const float* logp, const float* logp_rollout, const float* adv, const uint8_t* mask,
                        int64_t T, float eps_low, float eps_high, const int64_t* n_tokens, double* loss, float* g,
                        uint8_t* flags, int64_t* counts, hipStream_t st) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (st != nullptr) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(st, &sdev);
    if (e != hipSuccess) return e;
    if (sdev != dev) return hipErrorInvalidDevice;  // the stream must belong to the current device
  }
  // First call on this device (with it current): the device address of its copy.
  ScratchSlot& slot = g_scratch[dev];
  std::call_once(slot.once, [&] {
    void* p = nullptr;
    slot.err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (slot.err == hipSuccess) slot.ptr = p;
  });
  if (slot.err != hipSuccess) return slot.err;
  if (loss_layout(T).total > kLossScratchBytes) return hipErrorInvalidValue;  // the caller checked this
  // Every piece of the layout is written before it is read (block partials, then
  // the mask count when n_tokens is NULL), so nothing needs clearing between calls.
  return launch_loss(logp, logp_rollout, adv, mask, T, eps_low, eps_high, n_tokens, loss, g, flags, counts,
                     slot.ptr, st);
}

int launch_ppo_loss(const float* logp, const float* logp_old, const float* logp_behav, const float* adv,
                           const uint8_t* mask, int64_t T, float eps_low, float eps_high, const int64_t* n_tokens,
                           double* loss, float* g, uint8_t* flags, int64_t* counts, void* ws, hipStream_t st) {
  const LossLayout L = loss_layout(T);
  char* w8 = static_cast<char*>(ws);
  double* part_f = reinterpret_cast<double*>(w8 + L.part_f);
  int64_t* part_i = reinterpret_cast<int64_t*>(w8 + L.part_i);
  const int nblk = static_cast<int>(L.blocks);
  const int64_t* n_ptr = token_count(n_tokens, mask, T, L, w8, st);
  const bool vec_ok = aligned(logp, 16) && aligned(logp_old, 16) && aligned(logp_behav, 16) && aligned(adv, 16) &&
                      aligned(g, 16) && aligned(mask, 4) && aligned(flags, 4);
  if (logp_behav)
    hipLaunchKernelGGL(k_ppo<true>, dim3(nblk), dim3(kLossThreads), 0, st, logp, logp_old, logp_behav, adv, mask,
                       T, eps_low, eps_high, n_ptr, part_f, part_i, g, flags, vec_ok);
  else
    hipLaunchKernelGGL(k_ppo<false>, dim3(nblk), dim3(kLossThreads), 0, st, logp, logp_old, logp_behav, adv, mask,
                       T, eps_low, eps_high, n_ptr, part_f, part_i, g, flags, vec_ok);
  hipLaunchKernelGGL(k_loss_final, dim3(1), dim3(kLossThreads), 0, st, part_f, part_i, nblk, n_ptr, 1, loss,
                     counts);
  return hipGetLastError();
}

}  // namespace sao

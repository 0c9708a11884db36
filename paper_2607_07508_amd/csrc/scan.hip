// Skip-observation token-level GAE (Sec. 3.2, Eq. 4-5) as a segmented reverse scan.
//
// One workgroup per trajectory. Walking right to left, the state after a token is
//   s = (Vn, R, A, G): value of the next action, reward pending since the next
// action, and that action's advantage and return. Token t maps the state that
// enters from its right to the state that leaves to its left:
//   action (value v, reward r):  Vn' = v, R' = 0,
//                                A'  = (r + R) + gamma Vn - v + gamma lambda_b A,
//                                G'  = (r + R) + gamma G            (and A', G' are its outputs)
//   observation (reward r):      R' = R + r, everything else unchanged
// starting from s = 0 after the last token (no bootstrap after the last action;
// rewards before the first action leave through the left end and are dropped).
// Every such map, and every composition of them, has the form
//   Vn' = pV Vn + cV,  R' = pR R + cR,  A' = aV Vn + aR R + aA A + cA,  G' = gR R + gG G + cG,
// so a thread summarises its contiguous chunk by 11 numbers, the block scans the
// summaries (wave shuffles, then across waves through LDS), and each thread
// replays its chunk from the exact state that enters it. Arithmetic is float64.
#include "common.hpp"
#include "launch.hpp"
#include "../../include/sao.h"

namespace sao {

struct Aff {
  double pV, cV, pR, cR, aV, aR, aA, cA, gR, gG, cG;
};

__device__ __forceinline__ Aff aff_identity() {
  return Aff{1.0, 0.0, 1.0, 0.0, 0.0, 0.0, 1.0, 0.0, 0.0, 1.0, 0.0};
}

// (F o G)(s) = F(G(s)).
__device__ __forceinline__ Aff compose(const Aff& F, const Aff& G) {
  Aff r;
  r.pV = F.pV * G.pV;
  r.cV = fma(F.pV, G.cV, F.cV);
  r.pR = F.pR * G.pR;
  r.cR = fma(F.pR, G.cR, F.cR);
  r.aV = fma(F.aV, G.pV, F.aA * G.aV);
  r.aR = fma(F.aR, G.pR, F.aA * G.aR);
  r.aA = F.aA * G.aA;
  r.cA = fma(F.aV, G.cV, fma(F.aR, G.cR, fma(F.aA, G.cA, F.cA)));
  r.gR = fma(F.gR, G.pR, F.gG * G.gR);
  r.gG = F.gG * G.gG;
  r.cG = fma(F.gR, G.cR, fma(F.gG, G.cG, F.cG));
  return r;
}

__device__ __forceinline__ Aff token_map(bool action, double v, double r, double gamma, double kappa) {
  if (!action) {
    Aff m = aff_identity();
    m.cR = r;
    return m;
  }
  return Aff{0.0, v, 0.0, 0.0, gamma, 1.0, kappa, r - v, 1.0, gamma, r};
}

__device__ __forceinline__ Aff shfl_down_aff(const Aff& a, int d) {
  Aff o;
  o.pV = __shfl_down(a.pV, d, 64);
  o.cV = __shfl_down(a.cV, d, 64);
  o.pR = __shfl_down(a.pR, d, 64);
  o.cR = __shfl_down(a.cR, d, 64);
  o.aV = __shfl_down(a.aV, d, 64);
  o.aR = __shfl_down(a.aR, d, 64);
  o.aA = __shfl_down(a.aA, d, 64);
  o.cA = __shfl_down(a.cA, d, 64);
  o.gR = __shfl_down(a.gR, d, 64);
  o.gG = __shfl_down(a.gG, d, 64);
  o.cG = __shfl_down(a.cG, d, 64);
  return o;
}

// One block: cu_seqlens must rise from 0 to T without decreasing. Sets *bad (0/1),
// zeroes *n_tokens, and flags the status word.
__global__ __launch_bounds__(256) void k_check_segments(const int32_t* cu, int32_t B, int64_t T, int32_t* bad,
                                                        int64_t* n_tokens, int32_t* status) {
  __shared__ int32_t s_bad;
  if (threadIdx.x == 0) s_bad = (cu[0] != 0 || static_cast<int64_t>(cu[B]) != T) ? 1 : 0;
  __syncthreads();
  for (int32_t i = threadIdx.x; i < B; i += blockDim.x)
    if (cu[i + 1] < cu[i]) atomicOr(&s_bad, 1);
  __syncthreads();
  if (threadIdx.x == 0) {
    *bad = s_bad;
    if (n_tokens) *n_tokens = 0;
    if (s_bad && status) atomicOr(status, SAO_STATUS_SEGMENTS);
  }
}

constexpr int kScanThreads = 256;

__global__ __launch_bounds__(kScanThreads) void k_advantage(
    const float* values, const float* rewards, const uint8_t* mask, const int32_t* cu, int32_t B,
    int64_t T, double gamma, double lam, double alpha, float* adv, float* ret, int64_t* n_tokens,
    const int32_t* bad) {
  __shared__ Aff s_agg[kScanThreads / 64];
  __shared__ int64_t s_cnt[kScanThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  if (*bad) {
    // Malformed segments: every output is NaN; block b covers an even slice of [0, T).
    const int64_t lo = T * b / B, hi = T * (b + 1) / B;
    int64_t cnt = 0;
    for (int64_t t = lo + tid; t < hi; t += kScanThreads) {
      adv[t] = __builtin_nanf("");
      ret[t] = __builtin_nanf("");
      cnt += mask[t] != 0 ? 1 : 0;
    }
    cnt = wave_sum(cnt);
    if (lane == 0 && n_tokens && cnt)
      atomicAdd(reinterpret_cast<unsigned long long*>(n_tokens), static_cast<unsigned long long>(cnt));
    return;
  }
  const int64_t s = cu[b], e = cu[b + 1];
  const int64_t L = e - s;
  if (L == 0) return;
  double lam_b = lam;
  if (alpha > 0.0) {
    lam_b = 1.0 - 1.0 / (alpha * static_cast<double>(L));
    if (lam_b < 0.0) lam_b = 0.0;
  }
  const double kappa = gamma * lam_b;
  const int64_t chunk = (L + kScanThreads - 1) / kScanThreads;
  const int64_t c0 = s + tid * chunk;
  const int64_t c1 = c0 + chunk < e ? c0 + chunk : e;

  // Pass 1: this thread's chunk as one map, and its action count.
  Aff F = aff_identity();
  int64_t cnt = 0;
  for (int64_t t = c1 - 1; t >= c0; --t) {
    const bool act = mask[t] != 0;
    cnt += act ? 1 : 0;
    F = compose(token_map(act, values[t], rewards[t], gamma, kappa), F);
  }

  // Reverse inclusive scan inside the wave: P_l = F_l o F_{l+1} o ... o F_63.
  Aff P = F;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const Aff o = shfl_down_aff(P, d);
    if (lane + d < 64) P = compose(P, o);
  }
  const int64_t wcnt = wave_sum(cnt);
  if (lane == 0) {
    s_agg[wave] = P;
    s_cnt[wave] = wcnt;
  }
  __syncthreads();
  // State entering this wave from the right: later waves applied to the zero state.
  double sV = 0.0, sR = 0.0, sA = 0.0, sG = 0.0;
  for (int w = kScanThreads / 64 - 1; w > wave; --w) {
    const Aff& M = s_agg[w];
    const double nV = fma(M.pV, sV, M.cV);
    const double nR = fma(M.pR, sR, M.cR);
    const double nA = fma(M.aV, sV, fma(M.aR, sR, fma(M.aA, sA, M.cA)));
    const double nG = fma(M.gR, sR, fma(M.gG, sG, M.cG));
    sV = nV; sR = nR; sA = nA; sG = nG;
  }
  // State entering this thread: lanes to its right inside the wave, then the rest.
  const Aff Q = shfl_down_aff(P, 1);
  double Vn = sV, R = sR, A = sA, G = sG;
  if (lane < 63) {
    Vn = fma(Q.pV, sV, Q.cV);
    R = fma(Q.pR, sR, Q.cR);
    A = fma(Q.aV, sV, fma(Q.aR, sR, fma(Q.aA, sA, Q.cA)));
    G = fma(Q.gR, sR, fma(Q.gG, sG, Q.cG));
  }

  // Pass 2: replay the chunk from that state and write the outputs.
  for (int64_t t = c1 - 1; t >= c0; --t) {
    const double r = rewards[t];
    if (mask[t] != 0) {
      const double v = values[t];
      const double rt = r + R;
      const double An = fma(kappa, A, fma(gamma, Vn, rt - v));
      const double Gn = fma(gamma, G, rt);
      adv[t] = static_cast<float>(An);
      ret[t] = static_cast<float>(Gn);
      Vn = v;
      R = 0.0;
      A = An;
      G = Gn;
    } else {
      R += r;
      adv[t] = 0.0f;
      ret[t] = 0.0f;
    }
  }
  if (tid == 0 && n_tokens) {
    int64_t tot = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) tot += s_cnt[w];
    atomicAdd(reinterpret_cast<unsigned long long*>(n_tokens), static_cast<unsigned long long>(tot));
  }
}

hipError_t launch_advantage(const float* values, const float* rewards, const uint8_t* mask,
                            const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma, double lam,
                            double alpha, float* adv, float* ret, int64_t* n_tokens, int32_t* status,
                            void* ws, hipStream_t st) {
  int32_t* bad = static_cast<int32_t*>(ws);
  hipLaunchKernelGGL(k_check_segments, dim3(1), dim3(256), 0, st, cu_seqlens, B, T, bad, n_tokens, status);
  hipLaunchKernelGGL(k_advantage, dim3(B), dim3(kScanThreads), 0, st, values, rewards, mask, cu_seqlens,
                     B, T, gamma, lam, alpha, adv, ret, n_tokens, bad);
  return hipGetLastError();
}

}  // namespace sao

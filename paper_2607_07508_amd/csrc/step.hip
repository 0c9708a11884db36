// Step-level GAE (App. A.1): one advantage per agentic step.
//
// A step is a maximal run of loss-mask tokens inside a trajectory (one model
// turn). With steps [a_i, z_i), i < n, and a_n = the trajectory's end:
//   V_i = mean of values[a_i .. z_i)  or  values[z_i - 1]      (step average / last token)
//   R_i = sum of rewards[a_i .. a_{i+1})                       (observations fold into the step)
//   A_i = R_i + gamma V_{i+1} - V_i + gamma lambda_b A_{i+1},  G_i = R_i + gamma G_{i+1}
// with V_n = A_n = G_n = 0 and lambda_b = 1 - 1/(alpha n) when alpha > 0.
//
// One workgroup per trajectory, four phases separated by barriers:
//  1. left to right over 2048-token tiles: step starts and ends, numbered by a
//     block prefix count, go to a per-trajectory table in the workspace;
//  2. each wave reduces whole steps (values over the run, rewards over the run
//     and the observations after it) in a fixed lane order;
//  3. the recurrence over steps: each thread takes a contiguous chunk of steps,
//     summarises it as an affine map of the state entering from its right, one
//     thread chains the 256 maps, and each thread replays its chunk;
//  4. each wave writes its steps' tokens: A_i and G_i on the run, zeros on the
//     observations after it, and the step's last token in `last`.
// Arithmetic is float64; every reduction runs in a fixed order.
#include "common.hpp"
#include "launch.hpp"
#include "layout.hpp"
#include "segments.hpp"

namespace sao {

constexpr int kStepThreads = 256;
constexpr int kStepPer = 8;                               // tokens per thread per tile
constexpr int kStepTile = kStepThreads * kStepPer;

// Exclusive prefix sum over the block in thread order; *total gets the block's sum.
__device__ __forceinline__ int block_exclusive_scan(int x, int* sh, int* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int incl = x;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  __syncthreads();  // earlier readers of sh are done
  if (lane == 63) sh[wave] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kStepThreads / 64; ++w) {
    before += w < wave ? sh[w] : 0;
    all += sh[w];
  }
  *total = all;
  return before + incl - x;
}

__global__ __launch_bounds__(kStepThreads) void k_step_advantage(
    const float* values, const float* rewards, const uint8_t* mask, const int32_t* cu, int32_t B, int64_t T,
    double gamma, double lam, double alpha, bool last_value, float* adv, float* ret, uint8_t* last,
    int64_t* n_tokens, const int32_t* bad, int32_t* tab_a, int32_t* tab_z, double* tab_v, double* tab_r) {
  __shared__ int s_scan[kStepThreads / 64];
  __shared__ double s_map[kStepThreads][4];   // per chunk: A = cA + mA A_in, G = cG + mG G_in
  __shared__ double s_in[kStepThreads][2];    // (A, G) entering each chunk from the right
  __shared__ int64_t s_cnt[kStepThreads / 64];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b = blockIdx.x;
  if (*bad) {
    malformed_slice<kStepThreads>(mask, B, T, adv, ret, last, n_tokens);
    return;
  }
  const int64_t s = cu[b], e = cu[b + 1];
  const int64_t L = e - s;
  if (L <= 0) return;
  // The step table of this trajectory: entries [0, n) at offset s (n <= L).
  int32_t* ta = tab_a + s;
  int32_t* tz = tab_z + s;
  double* tv = tab_v + s;
  double* tr = tab_r + s;

  // Phase 1: step starts and ends (offsets from s), and the mask count.
  int n = 0, n_end = 0;
  int64_t cnt = 0;
  for (int64_t t0 = s / kStepTile * kStepTile; t0 < e; t0 += kStepTile) {
    const int64_t c0 = t0 + static_cast<int64_t>(tid) * kStepPer;
    bool m[kStepPer + 2];  // m[0] is token c0 - 1, m[kStepPer + 1] token c0 + kStepPer
#pragma unroll
    for (int j = 0; j < kStepPer + 2; ++j) {
      const int64_t t = c0 - 1 + j;
      m[j] = t >= s && t < e && mask[t] != 0;
    }
    int ns = 0, ne = 0;
#pragma unroll
    for (int j = 1; j <= kStepPer; ++j) {
      cnt += m[j] ? 1 : 0;
      ns += (m[j] && !m[j - 1]) ? 1 : 0;
      ne += (m[j] && !m[j + 1]) ? 1 : 0;
    }
    int tot_s, tot_e;
    int is = n + block_exclusive_scan(ns, s_scan, &tot_s);
    int ie = n_end + block_exclusive_scan(ne, s_scan, &tot_e);
#pragma unroll
    for (int j = 1; j <= kStepPer; ++j) {
      const int32_t off = static_cast<int32_t>(c0 - 1 + j - s);
      if (m[j] && !m[j - 1]) ta[is++] = off;
      if (m[j] && !m[j + 1]) tz[ie++] = off + 1;
    }
    n += tot_s;
    n_end += tot_e;
  }
  __syncthreads();  // the table is written (n_end == n: every run starts and ends)

  // Phase 2: V_i and R_i, one wave per step.
  for (int i = wave; i < n; i += kStepThreads / 64) {
    const int64_t a = ta[i], z = tz[i], nxt = i + 1 < n ? ta[i + 1] : L;
    double sv = 0.0, sr = 0.0;
    if (!last_value)
      for (int64_t t = a + lane; t < z; t += 64) sv += static_cast<double>(values[s + t]);
    for (int64_t t = a + lane; t < nxt; t += 64) sr += static_cast<double>(rewards[s + t]);
    sv = wave_sum(sv);
    sr = wave_sum(sr);
    if (lane == 0) {
      tv[i] = last_value ? static_cast<double>(values[s + z - 1]) : sv / static_cast<double>(z - a);
      tr[i] = sr;
    }
  }
  __syncthreads();

  // Phase 3: A_i and G_i. Thread j takes steps [p, q); its map sends the state
  // (A_q, G_q) entering from the right to (A_p, G_p).
  double lam_b = lam;
  if (alpha > 0.0) {
    lam_b = 1.0 - 1.0 / (alpha * static_cast<double>(n));
    if (lam_b < 0.0) lam_b = 0.0;
  }
  const double kappa = gamma * lam_b;
  const int per = (n + kStepThreads - 1) / kStepThreads;
  const int p = min(n, tid * per), q = min(n, p + per);
  const double v_right = q < n ? tv[q] : 0.0;   // read before any thread overwrites the table
  {
    double cA = 0.0, mA = 1.0, cG = 0.0, mG = 1.0, vn = v_right;
    for (int i = q - 1; i >= p; --i) {
      const double v = tv[i], r = tr[i];
      cA = fma(kappa, cA, fma(gamma, vn, r - v));
      mA *= kappa;
      cG = fma(gamma, cG, r);
      mG *= gamma;
      vn = v;
    }
    s_map[tid][0] = cA;
    s_map[tid][1] = mA;
    s_map[tid][2] = cG;
    s_map[tid][3] = mG;
  }
  __syncthreads();
  if (tid == 0) {
    double A = 0.0, G = 0.0;
    for (int j = kStepThreads - 1; j >= 0; --j) {
      s_in[j][0] = A;
      s_in[j][1] = G;
      A = fma(s_map[j][1], A, s_map[j][0]);
      G = fma(s_map[j][3], G, s_map[j][2]);
    }
  }
  __syncthreads();
  {
    double A = s_in[tid][0], G = s_in[tid][1], vn = v_right;
    for (int i = q - 1; i >= p; --i) {
      const double v = tv[i], r = tr[i];
      A = fma(kappa, A, fma(gamma, vn, r - v));
      G = fma(gamma, G, r);
      vn = v;
      tv[i] = A;  // the table now holds (A_i, G_i)
      tr[i] = G;
    }
  }
  __syncthreads();

  // Phase 4: outputs. Tokens before the first step, and every token of a
  // trajectory without steps, are zero; each wave then writes its steps' spans.
  const int64_t head = n > 0 ? ta[0] : L;
  for (int64_t t = tid; t < head; t += kStepThreads) {
    adv[s + t] = 0.0f;
    ret[s + t] = 0.0f;
    if (last) last[s + t] = 0;
  }
  for (int i = wave; i < n; i += kStepThreads / 64) {
    const int64_t a = ta[i], z = tz[i], nxt = i + 1 < n ? ta[i + 1] : L;
    const float A = static_cast<float>(tv[i]), G = static_cast<float>(tr[i]);
    for (int64_t t = a + lane; t < nxt; t += 64) {
      const bool in = t < z;
      adv[s + t] = in ? A : 0.0f;
      ret[s + t] = in ? G : 0.0f;
      if (last) last[s + t] = t == z - 1 ? 1 : 0;
    }
  }

  const int64_t wcnt = wave_sum(cnt);
  __syncthreads();
  if (lane == 0) s_cnt[wave] = wcnt;
  __syncthreads();
  if (tid == 0 && n_tokens) {
    int64_t tot = 0;
    for (int w = 0; w < kStepThreads / 64; ++w) tot += s_cnt[w];
    atomicAdd(reinterpret_cast<unsigned long long*>(n_tokens), static_cast<unsigned long long>(tot));
  }
}

hipError_t launch_step_advantage(const float* values, const float* rewards, const uint8_t* mask,
                                 const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma, double lam,
                                 double alpha, bool last_value, float* adv, float* ret, uint8_t* last,
                                 int64_t* n_tokens, int32_t* status, void* ws, hipStream_t st) {
  const StepLayout Ly = step_layout(T);
  char* w8 = static_cast<char*>(ws);
  int32_t* bad = reinterpret_cast<int32_t*>(w8 + Ly.bad);
  hipLaunchKernelGGL(k_check_segments<256>, dim3(1), dim3(256), 0, st, cu_seqlens, B, T, bad, n_tokens, status);
  hipLaunchKernelGGL(k_step_advantage, dim3(B), dim3(kStepThreads), 0, st, values, rewards, mask, cu_seqlens, B, T,
                     gamma, lam, alpha, last_value, adv, ret, last, n_tokens, bad,
                     reinterpret_cast<int32_t*>(w8 + Ly.tab_a), reinterpret_cast<int32_t*>(w8 + Ly.tab_z),
                     reinterpret_cast<double*>(w8 + Ly.tab_v), reinterpret_cast<double*>(w8 + Ly.tab_r));
  return hipGetLastError();
}

}  // namespace sao

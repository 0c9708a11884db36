// Critic-free advantage baselines the paper compares with, one advantage per
// trajectory, placed on every loss-mask token of it:
//  * GRPO's group normalisation (Sec. 2): trajectories [g G, (g+1) G) answer one
//    prompt, A_b = (R_b - mu_g) / sqrt(var_g + eps_stab) with population variance;
//  * a running-mean reward baseline (the 8 most recent rewards of each prompt in
//    the Sec. 4.3 ablation, the 128 most recent in the Sec. 4.5 online
//    comparison): A_b = R_b - mean of the `window` most recent earlier rewards
//    of b's key, the caller's history first and then the batch in order.
// R_b is the sum of trajectory b's token rewards. Sums are float64 in a fixed
// order. The batch has few trajectories (one per rollout), so the per-trajectory
// kernels use one thread per trajectory and the per-token work one workgroup per
// trajectory.
#include "common.hpp"
#include "launch.hpp"
#include "reduce.hpp"
#include "segments.hpp"

namespace sao {

constexpr int kBaseThreads = 256;

// R_b (one workgroup per trajectory) and the loss-mask count. With malformed
// segments every R_b is NaN and the count is left to the broadcast.
__global__ __launch_bounds__(kBaseThreads) void k_traj_reward(const float* rewards, const uint8_t* mask,
                                                              const int32_t* cu, const int32_t* bad, double* R,
                                                              int64_t* n_tokens) {
  __shared__ double shd[kBaseThreads / 64];
  __shared__ int64_t shi[kBaseThreads / 64];
  const int b = blockIdx.x;
  if (*bad) {
    if (threadIdx.x == 0) R[b] = __builtin_nan("");
    return;
  }
  const int64_t s = cu[b], e = cu[b + 1];
  double acc = 0.0;
  int64_t cnt = 0;
  for (int64_t t = s + threadIdx.x; t < e; t += kBaseThreads) {
    acc += static_cast<double>(rewards[t]);
    cnt += mask[t] != 0 ? 1 : 0;
  }
  acc = block_sum<kBaseThreads>(acc, shd);
  cnt = block_sum<kBaseThreads>(cnt, shi);
  if (threadIdx.x == 0) {
    R[b] = acc;
    if (n_tokens && cnt) atomicAdd(reinterpret_cast<unsigned long long*>(n_tokens), static_cast<unsigned long long>(cnt));
  }
}

// GRPO: one thread per trajectory; its group's mean and variance in member order.
__global__ __launch_bounds__(kBaseThreads) void k_group_adv(const double* R, int32_t B, int32_t G, double eps_stab,
                                                            double* A) {
  const int b = blockIdx.x * kBaseThreads + threadIdx.x;
  if (b >= B) return;
  const int g0 = b / G * G;
  double mu = 0.0;
  for (int j = 0; j < G; ++j) mu += R[g0 + j];
  mu /= static_cast<double>(G);
  double var = 0.0;
  for (int j = 0; j < G; ++j) {
    const double d = R[g0 + j] - mu;
    var = fma(d, d, var);
  }
  var /= static_cast<double>(G);
  A[b] = (R[b] - mu) / sqrt(var + eps_stab);
}

// The key of trajectory b (0 without keys), or -1 if it is out of range.
__device__ __forceinline__ int32_t key_of(const int32_t* keys, int32_t n_keys, int b) {
  if (!keys) return 0;
  const int32_t k = keys[b];
  return (k >= 0 && k < n_keys) ? k : -1;
}

// Running mean: one thread per trajectory. The window is filled from the most
// recent earlier same-key trajectories of the batch, then from the history ring
// (hist[k][slot], slot = position mod window; seen[k] rewards pushed so far).
__global__ __launch_bounds__(kBaseThreads) void k_running_mean(const double* R, int32_t B, const int32_t* keys,
                                                               int32_t n_keys, int32_t window, const double* hist,
                                                               const int64_t* seen, const int32_t* bad, double* A,
                                                               int32_t* status) {
  const int b = blockIdx.x * kBaseThreads + threadIdx.x;
  if (b >= B) return;
  if (*bad) {
    A[b] = __builtin_nan("");
    return;
  }
  const int32_t k = key_of(keys, n_keys, b);
  if (k < 0) {
    A[b] = __builtin_nan("");
    if (status) atomicOr(status, SAO_STATUS_KEY_RANGE);
    return;
  }
  double sum = 0.0;
  int64_t c = 0;
  for (int j = b - 1; j >= 0 && c < window; --j) {
    if (key_of(keys, n_keys, j) != k) continue;
    sum += R[j];
    ++c;
  }
  const int64_t h = seen[k];
  const double* ring = hist + static_cast<int64_t>(k) * window;
  for (int64_t i = 0; i < h && c < window; ++i, ++c) sum += ring[(h - 1 - i) % window];
  A[b] = R[b] - (c > 0 ? sum / static_cast<double>(c) : 0.0);
}

// Pushes the batch's rewards into the rings: trajectory b of rank r among its
// key's n trajectories (in order) lands in slot (seen + r) mod window if it is
// one of the last `window` of them. seen itself moves in k_seen_update.
__global__ __launch_bounds__(kBaseThreads) void k_history_update(const double* R, int32_t B, const int32_t* keys,
                                                                 int32_t n_keys, int32_t window, double* hist,
                                                                 const int64_t* seen, const int32_t* bad) {
  const int b = blockIdx.x * kBaseThreads + threadIdx.x;
  if (b >= B || *bad) return;
  const int32_t k = key_of(keys, n_keys, b);
  if (k < 0) return;
  int64_t rank = 0, cnt = 0;
  if (!keys) {
    rank = b;
    cnt = B;
  } else {
    for (int j = 0; j < B; ++j) {
      if (key_of(keys, n_keys, j) != k) continue;
      rank += j < b ? 1 : 0;
      ++cnt;
    }
  }
  if (rank >= cnt - window) hist[static_cast<int64_t>(k) * window + (seen[k] + rank) % window] = R[b];
}

// seen[k] += number of the batch's trajectories with key k (one thread per key).
__global__ __launch_bounds__(kBaseThreads) void k_seen_update(int32_t B, const int32_t* keys, int32_t n_keys,
                                                              int64_t* seen, const int32_t* bad) {
  const int k = blockIdx.x * kBaseThreads + threadIdx.x;
  if (k >= n_keys || *bad) return;
  int64_t cnt = 0;
  if (!keys)
    cnt = B;
  else
    for (int j = 0; j < B; ++j) cnt += key_of(keys, n_keys, j) == k ? 1 : 0;
  seen[k] += cnt;
}

// adv[t] = A_b on trajectory b's loss-mask tokens, 0 elsewhere (one workgroup per
// trajectory); NaN everywhere with malformed segments.
__global__ __launch_bounds__(kBaseThreads) void k_broadcast(const uint8_t* mask, const int32_t* cu, int32_t B,
                                                            int64_t T, const double* A, const int32_t* bad,
                                                            float* adv, int64_t* n_tokens) {
  if (*bad) {
    malformed_slice<kBaseThreads>(mask, B, T, adv, nullptr, nullptr, n_tokens);
    return;
  }
  const int b = blockIdx.x;
  const int64_t s = cu[b], e = cu[b + 1];
  const float a = static_cast<float>(A[b]);
  for (int64_t t = s + threadIdx.x; t < e; t += kBaseThreads) adv[t] = mask[t] != 0 ? a : 0.0f;
}

namespace {
inline unsigned blocks_for(int64_t n) { return static_cast<unsigned>((n + kBaseThreads - 1) / kBaseThreads); }
}  // namespace

hipError_t launch_group_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens, int32_t B,
                                  int64_t T, int32_t group_size, double eps_stab, float* adv, double* traj_reward,
                                  double* traj_adv, int64_t* n_tokens, int32_t* status, void* ws, hipStream_t st) {
  int32_t* bad = static_cast<int32_t*>(ws);
  hipLaunchKernelGGL(k_check_segments<256>, dim3(1), dim3(256), 0, st, cu_seqlens, B, T, bad, n_tokens, status);
  hipLaunchKernelGGL(k_traj_reward, dim3(B), dim3(kBaseThreads), 0, st, rewards, mask, cu_seqlens, bad, traj_reward,
                     n_tokens);
  hipLaunchKernelGGL(k_group_adv, dim3(blocks_for(B)), dim3(kBaseThreads), 0, st, traj_reward, B, group_size,
                     eps_stab, traj_adv);
  hipLaunchKernelGGL(k_broadcast, dim3(B), dim3(kBaseThreads), 0, st, mask, cu_seqlens, B, T, traj_adv, bad, adv,
                     n_tokens);
  return hipGetLastError();
}

hipError_t launch_running_mean_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens,
                                         int32_t B, int64_t T, const int32_t* keys, int32_t n_keys, int32_t window,
                                         double* history, int64_t* seen, float* adv, double* traj_reward,
                                         double* traj_adv, int64_t* n_tokens, int32_t* status, void* ws,
                                         hipStream_t st) {
  int32_t* bad = static_cast<int32_t*>(ws);
  hipLaunchKernelGGL(k_check_segments<256>, dim3(1), dim3(256), 0, st, cu_seqlens, B, T, bad, n_tokens, status);
  hipLaunchKernelGGL(k_traj_reward, dim3(B), dim3(kBaseThreads), 0, st, rewards, mask, cu_seqlens, bad, traj_reward,
                     n_tokens);
  hipLaunchKernelGGL(k_running_mean, dim3(blocks_for(B)), dim3(kBaseThreads), 0, st, traj_reward, B, keys, n_keys,
                     window, history, seen, bad, traj_adv, status);
  hipLaunchKernelGGL(k_history_update, dim3(blocks_for(B)), dim3(kBaseThreads), 0, st, traj_reward, B, keys, n_keys,
                     window, history, seen, bad);
  hipLaunchKernelGGL(k_seen_update, dim3(blocks_for(n_keys)), dim3(kBaseThreads), 0, st, B, keys, n_keys, seen, bad);
  hipLaunchKernelGGL(k_broadcast, dim3(B), dim3(kBaseThreads), 0, st, mask, cu_seqlens, B, T, traj_adv, bad, adv,
                     n_tokens);
  return hipGetLastError();
}

}  // namespace sao

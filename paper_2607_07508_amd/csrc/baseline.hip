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
#include "layout.hpp"
#include "reduce.hpp"
#include "segments.hpp"

namespace sao {

constexpr int kBaseThreads = 256;

// [s, e) as a scalar head, a body of whole aligned groups of 4 tokens, and a
// scalar tail; body(t) handles tokens t .. t+3 with 16-byte (float) and 4-byte
// (mask) vector access, one(t) a single token. Block threads stride the body.
template <class Body, class One>
__device__ __forceinline__ void walk_span(int64_t s, int64_t e, bool vec_ok, Body&& body, One&& one) {
  const int64_t b0 = vec_ok ? min(e, (s + 3) / 4 * 4) : e;
  const int64_t b1 = vec_ok ? max(b0, e / 4 * 4) : e;
  for (int64_t t = s + threadIdx.x; t < b0; t += kBaseThreads) one(t);
  // Unrolled so that a thread's loads of successive blocks are in flight together;
  // the bodies still run, and accumulate, in token order.
#pragma unroll 4
  for (int64_t t = b0 + 4 * static_cast<int64_t>(threadIdx.x); t < b1; t += 4 * kBaseThreads) body(t);
  for (int64_t t = b1 + threadIdx.x; t < e; t += kBaseThreads) one(t);
}

// R_b, one workgroup per trajectory; NaN for every b with malformed segments.
__global__ __launch_bounds__(kBaseThreads) void k_traj_reward(const float* rewards, const int32_t* cu,
                                                              const int32_t* bad, double* R, bool vec_ok) {
  __shared__ double shd[kBaseThreads / 64];
  const int b = blockIdx.x;
  if (*bad) {
    if (threadIdx.x == 0) R[b] = __builtin_nan("");
    return;
  }
  double acc = 0.0;
  walk_span(
      cu[b], cu[b + 1], vec_ok,
      [&](int64_t t) {
        const f32x4_t r4 = *reinterpret_cast<const f32x4_t*>(rewards + t);
        acc += (static_cast<double>(r4[0]) + static_cast<double>(r4[1])) +
               (static_cast<double>(r4[2]) + static_cast<double>(r4[3]));
      },
      [&](int64_t t) { acc += static_cast<double>(rewards[t]); });
  acc = block_sum<kBaseThreads>(acc, shd);
  if (threadIdx.x == 0) R[b] = acc;
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

// Running mean: one wave per trajectory. The window is filled from the most
// recent earlier same-key trajectories of the batch, 64 candidates at a time
// (a ballot ranks the matches), then from the history ring (hist[k][slot],
// slot = position mod window; seen[k] rewards pushed so far). Lane partial sums
// are added in lane order.
__global__ __launch_bounds__(kBaseThreads) void k_running_mean(const double* R, int32_t B, const int32_t* keys,
                                                               int32_t n_keys, int32_t window, const double* hist,
                                                               const int64_t* seen, const int32_t* bad, double* A,
                                                               int32_t* status) {
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.x * (kBaseThreads / 64) + (threadIdx.x >> 6);
  if (b >= B) return;
  if (*bad) {
    if (lane == 0) A[b] = __builtin_nan("");
    return;
  }
  const int32_t k = key_of(keys, n_keys, b);
  if (k < 0) {
    if (lane == 0) {
      A[b] = __builtin_nan("");
      if (status) atomicOr(status, SAO_STATUS_KEY_RANGE);
    }
    return;
  }
  double sum = 0.0;
  int64_t c = 0;  // matches found so far (uniform across the wave)
  const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
  for (int j0 = b - 1; j0 >= 0 && c < window; j0 -= 64) {
    const int j = j0 - lane;  // lane 0 is the most recent candidate
    const bool match = j >= 0 && key_of(keys, n_keys, j) == k;
    const uint64_t ballot = __ballot(match);
    const int64_t rank = c + __popcll(ballot & below);
    if (match && rank < window) sum += R[j];
    c += __popcll(ballot);
  }
  const int64_t in_batch = c < window ? c : window;
  const int64_t h = seen[k];
  const int64_t from_hist = min(h, static_cast<int64_t>(window) - in_batch);
  const double* ring = hist + static_cast<int64_t>(k) * window;
  for (int64_t i = lane; i < from_hist; i += 64) sum += ring[(h - 1 - i) % window];
  sum = wave_sum(sum);
  const int64_t cnt = in_batch + from_hist;
  if (lane == 0) A[b] = R[b] - (cnt > 0 ? sum / static_cast<double>(cnt) : 0.0);
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
// trajectory), and the loss-mask count into the count slots; NaN everywhere with
// malformed segments.
__global__ __launch_bounds__(kBaseThreads) void k_broadcast(const uint8_t* mask, const int32_t* cu, int32_t B,
                                                            int64_t T, const double* A, const int32_t* bad,
                                                            float* adv, int64_t* slots, bool vec_ok) {
  if (*bad) {
    malformed_slice<kBaseThreads, kCountSlots>(mask, B, T, adv, nullptr, nullptr, slots);
    return;
  }
  __shared__ int64_t shi[kBaseThreads / 64];
  const int b = blockIdx.x;
  const float a = static_cast<float>(A[b]);
  int64_t cnt = 0;
  walk_span(
      cu[b], cu[b + 1], vec_ok,
      [&](int64_t t) {
        const uint32_t m4 = *reinterpret_cast<const uint32_t*>(mask + t);
        const bool m0 = (m4 & 0xffu) != 0, m1 = (m4 & 0xff00u) != 0, m2 = (m4 & 0xff0000u) != 0,
                   m3 = (m4 & 0xff000000u) != 0;
        *reinterpret_cast<f32x4_t*>(adv + t) = f32x4_t{m0 ? a : 0.0f, m1 ? a : 0.0f, m2 ? a : 0.0f, m3 ? a : 0.0f};
        cnt += static_cast<int64_t>(m0) + m1 + m2 + m3;
      },
      [&](int64_t t) {
        const bool m = mask[t] != 0;
        adv[t] = m ? a : 0.0f;
        cnt += m ? 1 : 0;
      });
  cnt = block_sum<kBaseThreads>(cnt, shi);
  if (threadIdx.x == 0) add_count<kCountSlots>(slots, cnt);
}

namespace {
inline unsigned blocks_for(int64_t n) { return static_cast<unsigned>((n + kBaseThreads - 1) / kBaseThreads); }

// Vector access needs 16-byte aligned float arrays and a 4-byte aligned mask.
bool span_vec_ok(const float* rewards, const uint8_t* mask, const float* adv) {
  return ((reinterpret_cast<uintptr_t>(rewards) | reinterpret_cast<uintptr_t>(adv)) & 15u) == 0 &&
         (reinterpret_cast<uintptr_t>(mask) & 3u) == 0;
}
}  // namespace

int launch_group_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens, int32_t B,
                                  int64_t T, int32_t group_size, double eps_stab, float* adv, double* traj_reward,
                                  double* traj_adv, int64_t* n_tokens, int32_t* status, void* ws, hipStream_t st) {
  const SegHead H = seg_head();
  char* w8 = static_cast<char*>(ws);
  int32_t* bad = reinterpret_cast<int32_t*>(w8 + H.bad);
  int64_t* slots = reinterpret_cast<int64_t*>(w8 + H.slots);
  hipLaunchKernelGGL((k_check_segments<256, kCountSlots>), dim3(1), dim3(256), 0, st, cu_seqlens, B, T, bad, slots,
                     status);
  const bool vec_ok = span_vec_ok(rewards, mask, adv);
  hipLaunchKernelGGL(k_traj_reward, dim3(B), dim3(kBaseThreads), 0, st, rewards, cu_seqlens, bad, traj_reward,
                     vec_ok);
  hipLaunchKernelGGL(k_group_adv, dim3(blocks_for(B)), dim3(kBaseThreads), 0, st, traj_reward, B, group_size,
                     eps_stab, traj_adv);
  hipLaunchKernelGGL(k_broadcast, dim3(B), dim3(kBaseThreads), 0, st, mask, cu_seqlens, B, T, traj_adv, bad, adv,
                     slots, vec_ok);
  if (n_tokens) hipLaunchKernelGGL(k_slots_total<kCountSlots>, dim3(1), dim3(64), 0, st, slots, n_tokens);
  return hipGetLastError();
}

int launch_running_mean_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens,
                                         int32_t B, int64_t T, const int32_t* keys, int32_t n_keys, int32_t window,
                                         double* history, int64_t* seen, float* adv, double* traj_reward,
                                         double* traj_adv, int64_t* n_tokens, int32_t* status, void* ws,
                                         hipStream_t st) {
  const SegHead H = seg_head();
  char* w8 = static_cast<char*>(ws);
  int32_t* bad = reinterpret_cast<int32_t*>(w8 + H.bad);
  int64_t* slots = reinterpret_cast<int64_t*>(w8 + H.slots);
  hipLaunchKernelGGL((k_check_segments<256, kCountSlots>), dim3(1), dim3(256), 0, st, cu_seqlens, B, T, bad, slots,
                     status);
  const bool vec_ok = span_vec_ok(rewards, mask, adv);
  hipLaunchKernelGGL(k_traj_reward, dim3(B), dim3(kBaseThreads), 0, st, rewards, cu_seqlens, bad, traj_reward,
                     vec_ok);
  hipLaunchKernelGGL(k_running_mean, dim3(blocks_for(64 * static_cast<int64_t>(B))), dim3(kBaseThreads), 0, st,
                     traj_reward, B, keys, n_keys, window, history, seen, bad, traj_adv, status);
  hipLaunchKernelGGL(k_history_update, dim3(blocks_for(B)), dim3(kBaseThreads), 0, st, traj_reward, B, keys, n_keys,
                     window, history, seen, bad);
  hipLaunchKernelGGL(k_seen_update, dim3(blocks_for(n_keys)), dim3(kBaseThreads), 0, st, B, keys, n_keys, seen, bad);
  hipLaunchKernelGGL(k_broadcast, dim3(B), dim3(kBaseThreads), 0, st, mask, cu_seqlens, B, T, traj_adv, bad, adv,
                     slots, vec_ok);
  if (n_tokens) hipLaunchKernelGGL(k_slots_total<kCountSlots>, dim3(1), dim3(64), 0, st, slots, n_tokens);
  return hipGetLastError();
}

}  // namespace sao

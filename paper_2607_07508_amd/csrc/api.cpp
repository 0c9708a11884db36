// C ABI of the SAO loss pass: host-side validation, workspace sizing, dispatch to
// the launchers. Every check below runs before any HIP call, so argument errors
// never touch the device. This translation unit includes no HIP header: it builds
// with a plain host compiler too, which is how the validation layer is run under
// the address and undefined-behaviour sanitizers on a machine without a GPU.
#include <cmath>
#include <cstdarg>
#include <cstdio>

#include "../../include/sao.h"
#include "launch.hpp"
#include "layout.hpp"

namespace {

thread_local char g_msg[512] = "";

sao_status_t fail(sao_status_t s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return s;
}

sao_status_t ok() {
  g_msg[0] = '\0';
  return SAO_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t esize_of(sao_dtype_t d) { return d == SAO_BF16 ? 2 : 4; }

constexpr int64_t kMaxRows = (int64_t{1} << 31) - 1024;
// The MFMA tile engine forms each lane's copy offset in 32 bits as
// row * ld * element size with row < 256, so a row stride may span at most 2^24 bytes.
constexpr int64_t kMaxRowBytes = int64_t{1} << 24;

sao_status_t check_head(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w, int64_t T,
                        int64_t H, int64_t V, sao_dtype_t dtype) {
  if (dtype != SAO_BF16 && dtype != SAO_F32) return fail(SAO_ERR_DTYPE, "unknown dtype %d", (int)dtype);
  if (T < 0 || T > kMaxRows) return fail(SAO_ERR_SHAPE, "T=%lld out of range", (long long)T);
  if (H < 8 || H % 8 != 0) return fail(SAO_ERR_SHAPE, "H=%lld must be a positive multiple of 8", (long long)H);
  if (V < 1 || V > kMaxRows) return fail(SAO_ERR_SHAPE, "V=%lld out of range", (long long)V);
  if (ld_hidden < H || ld_hidden % 8 != 0)
    return fail(SAO_ERR_SHAPE, "ld_hidden=%lld must be >= H and a multiple of 8", (long long)ld_hidden);
  if (ld_w < H || ld_w % 8 != 0)
    return fail(SAO_ERR_SHAPE, "ld_w=%lld must be >= H and a multiple of 8", (long long)ld_w);
  const int64_t es = static_cast<int64_t>(esize_of(dtype));
  if (ld_hidden > kMaxRowBytes / es || ld_w > kMaxRowBytes / es)
    return fail(SAO_ERR_SHAPE, "ld_hidden=%lld, ld_w=%lld: row strides are limited to %lld elements",
                (long long)ld_hidden, (long long)ld_w, (long long)(kMaxRowBytes / es));
  if (!aligned16(hidden) || !aligned16(w_head))
    return fail(SAO_ERR_SHAPE, "hidden and w_head must be 16-byte aligned");
  return SAO_OK;
}

sao_status_t check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return SAO_OK;
  if (!ws) return fail(SAO_ERR_NULL, "workspace of %zu bytes required", need);
  if (ws_bytes < need) return fail(SAO_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need);
  if ((reinterpret_cast<uintptr_t>(ws) & 255u) != 0) return fail(SAO_ERR_WORKSPACE, "workspace not 256-byte aligned");
  return SAO_OK;
}

// Checks shared by the advantage entry points.
sao_status_t check_segments_args(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens, int32_t B,
                                 int64_t T, const float* adv) {
  if (!rewards || !mask || !cu_seqlens || !adv) return fail(SAO_ERR_NULL, "rewards, mask, cu_seqlens and adv are required");
  if (B < 1) return fail(SAO_ERR_SHAPE, "B=%d must be >= 1", (int)B);
  if (T < 0 || T > kMaxRows) return fail(SAO_ERR_SHAPE, "T=%lld out of range", (long long)T);
  return SAO_OK;
}

sao_status_t device(int e, const char* what) {
  if (e != 0) return fail(SAO_ERR_DEVICE, "%s: %s", what, sao::device_error_string(e));
  return ok();
}

// alpha > 0 selects the length-adaptive lambda, alpha == 0 the fixed one.
sao_status_t check_discounts(double gamma, double lam, double alpha) {
  if (!(gamma >= 0.0 && gamma <= 1.0)) return fail(SAO_ERR_VALUE, "gamma=%g outside [0,1]", gamma);
  if (!(lam >= 0.0 && lam <= 1.0)) return fail(SAO_ERR_VALUE, "lam=%g outside [0,1]", lam);
  if (!std::isfinite(alpha) || alpha < 0.0) return fail(SAO_ERR_VALUE, "alpha=%g must be finite and >= 0", alpha);
  return SAO_OK;
}

}  // namespace

extern "C" {

const char* sao_status_string(sao_status_t s) {
  switch (s) {
    case SAO_OK: return "ok";
    case SAO_ERR_NULL: return "null pointer";
    case SAO_ERR_SHAPE: return "bad shape";
    case SAO_ERR_VALUE: return "bad value";
    case SAO_ERR_DTYPE: return "bad dtype";
    case SAO_ERR_WORKSPACE: return "workspace too small";
    case SAO_ERR_DEVICE: return "device error";
  }
  return "unknown status";
}

const char* sao_last_error_message(void) { return g_msg; }

const char* sao_version(void) { return "0.1.0"; }

size_t sao_workspace_size(sao_op_t op, int64_t T, int64_t H, int64_t V, sao_dtype_t dtype) {
  if (T < 0 || (dtype != SAO_BF16 && dtype != SAO_F32)) return 0;
  if (T == 0) return 0;
  switch (op) {
    case SAO_OP_LOGPROB:
      if (H < 1 || V < 1) return 0;
      return sao::logprob_layout(T, H, V, esize_of(dtype)).total;
    case SAO_OP_BACKWARD:
      if (H < 1 || V < 1) return 0;
      return sao::backward_layout(T, H, V, esize_of(dtype)).total;
    case SAO_OP_LOSS:
      return sao::loss_layout(T).total;
    case SAO_OP_ADVANTAGE:
      return sao::advantage_workspace();
    case SAO_OP_VALUE:
      if (H < 1) return 0;
      return sao::value_layout(T, H).total;
    case SAO_OP_PPO_LOSS:
      return sao::loss_layout(T).total;
    case SAO_OP_EXPLAINED_VARIANCE:
      return sao::ev_layout(T).total;
    case SAO_OP_STEP_ADVANTAGE:
      return sao::step_layout(T).total;
    case SAO_OP_GROUP_ADVANTAGE:
    case SAO_OP_RUNNING_MEAN_ADVANTAGE:
      return sao::advantage_workspace();
  }
  return 0;
}

sao_status_t sao_token_logprob(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w,
                               const int32_t* target, const uint8_t* mask, int64_t T, int64_t H, int64_t V,
                               sao_dtype_t dtype, float* logp, float* lse, int32_t* status, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  if (!hidden || !w_head || !target || !logp || !lse)
    return fail(SAO_ERR_NULL, "hidden, w_head, target, logp and lse are required");
  if (sao_status_t s = check_head(hidden, ld_hidden, w_head, ld_w, T, H, V, dtype)) return s;
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_LOGPROB, T, H, V, dtype))) return s;
  return device(sao::launch_logprob(hidden, ld_hidden, w_head, ld_w, target, mask, T, H, V, dtype == SAO_BF16,
                                    logp, lse, status, ws, stream),
                "sao_token_logprob launch");
}

sao_status_t sao_advantage(const float* values, const float* rewards, const uint8_t* mask,
                           const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma, double lam,
                           double alpha, float* adv, float* ret, int64_t* n_tokens, int32_t* status, void* ws,
                           size_t ws_bytes, hipStream_t stream) {
  if (!values || !rewards || !mask || !cu_seqlens || !adv || !ret)
    return fail(SAO_ERR_NULL, "values, rewards, mask, cu_seqlens, adv and ret are required");
  if (B < 1) return fail(SAO_ERR_SHAPE, "B=%d must be >= 1", (int)B);
  if (T < 0 || T > kMaxRows) return fail(SAO_ERR_SHAPE, "T=%lld out of range", (long long)T);
  if (sao_status_t s = check_discounts(gamma, lam, alpha)) return s;
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_ADVANTAGE, T, 1, 1, SAO_F32))) return s;
  return device(sao::launch_advantage(values, rewards, mask, cu_seqlens, B, T, gamma, lam, alpha, adv, ret,
                                      n_tokens, status, ws, stream),
                "sao_advantage launch");
}

sao_status_t sao_step_advantage(const float* values, const float* rewards, const uint8_t* mask,
                                const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma, double lam,
                                double alpha, sao_step_value_t step_value, float* adv, float* ret, uint8_t* last,
                                int64_t* n_tokens, int32_t* status, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!values || !rewards || !mask || !cu_seqlens || !adv || !ret)
    return fail(SAO_ERR_NULL, "values, rewards, mask, cu_seqlens, adv and ret are required");
  if (B < 1) return fail(SAO_ERR_SHAPE, "B=%d must be >= 1", (int)B);
  if (T < 0 || T > kMaxRows) return fail(SAO_ERR_SHAPE, "T=%lld out of range", (long long)T);
  if (sao_status_t s = check_discounts(gamma, lam, alpha)) return s;
  if (step_value != SAO_STEP_AVERAGE && step_value != SAO_STEP_LAST)
    return fail(SAO_ERR_VALUE, "unknown step value form %d", (int)step_value);
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_STEP_ADVANTAGE, T, 1, 1, SAO_F32)))
    return s;
  return device(sao::launch_step_advantage(values, rewards, mask, cu_seqlens, B, T, gamma, lam, alpha,
                                           step_value == SAO_STEP_LAST, adv, ret, last, n_tokens, status, ws,
                                           stream),
                "sao_step_advantage launch");
}

sao_status_t sao_group_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens, int32_t B,
                                 int64_t T, int32_t group_size, double eps_stab, float* adv, double* traj_reward,
                                 double* traj_adv, int64_t* n_tokens, int32_t* status, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  if (sao_status_t s = check_segments_args(rewards, mask, cu_seqlens, B, T, adv)) return s;
  if (!traj_reward || !traj_adv) return fail(SAO_ERR_NULL, "traj_reward and traj_adv are required");
  if (group_size < 1 || B % group_size != 0)
    return fail(SAO_ERR_SHAPE, "B=%d must be a positive multiple of group_size=%d", (int)B, (int)group_size);
  if (!(eps_stab >= 0.0) || !std::isfinite(eps_stab)) return fail(SAO_ERR_VALUE, "eps_stab must be finite and >= 0");
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_GROUP_ADVANTAGE, T, 1, 1, SAO_F32))) return s;
  return device(sao::launch_group_advantage(rewards, mask, cu_seqlens, B, T, group_size, eps_stab, adv, traj_reward,
                                            traj_adv, n_tokens, status, ws, stream),
                "sao_group_advantage launch");
}

sao_status_t sao_running_mean_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens,
                                        int32_t B, int64_t T, const int32_t* keys, int32_t n_keys, int32_t window,
                                        double* history, int64_t* seen, float* adv, double* traj_reward,
                                        double* traj_adv, int64_t* n_tokens, int32_t* status, void* ws,
                                        size_t ws_bytes, hipStream_t stream) {
  if (sao_status_t s = check_segments_args(rewards, mask, cu_seqlens, B, T, adv)) return s;
  if (!traj_reward || !traj_adv || !history || !seen)
    return fail(SAO_ERR_NULL, "traj_reward, traj_adv, history and seen are required");
  if (n_keys < 1) return fail(SAO_ERR_SHAPE, "n_keys=%d must be >= 1", (int)n_keys);
  if (window < 1) return fail(SAO_ERR_SHAPE, "window=%d must be >= 1", (int)window);
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_RUNNING_MEAN_ADVANTAGE, T, 1, 1, SAO_F32)))
    return s;
  return device(sao::launch_running_mean_advantage(rewards, mask, cu_seqlens, B, T, keys, n_keys, window, history,
                                                   seen, adv, traj_reward, traj_adv, n_tokens, status, ws, stream),
                "sao_running_mean_advantage launch");
}

sao_status_t sao_clipped_loss(const float* logp, const float* logp_rollout, const float* adv,
                              const uint8_t* mask, int64_t T, float eps_low, float eps_high,
                              const int64_t* n_tokens, double* loss, float* g, uint8_t* flags, int64_t* counts,
                              void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!logp || !logp_rollout || !adv || !mask || !loss || !g || !flags || !counts)
    return fail(SAO_ERR_NULL, "logp, logp_rollout, adv, mask, loss, g, flags and counts are required");
  if (T < 0 || T > kMaxRows) return fail(SAO_ERR_SHAPE, "T=%lld out of range", (long long)T);
  if (!(eps_low >= 0.0f) || !std::isfinite(eps_low) || !(eps_high >= 0.0f) || !std::isfinite(eps_high))
    return fail(SAO_ERR_VALUE, "eps_low=%g, eps_high=%g must be finite and >= 0", eps_low, eps_high);
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_LOSS, T, 1, 1, SAO_F32))) return s;
  return device(sao::launch_loss(logp, logp_rollout, adv, mask, T, eps_low, eps_high, n_tokens, loss, g, flags,
                                 counts, ws, stream),
                "sao_clipped_loss launch");
}

sao_status_t sao_clipped_loss_noalloc(const float* logp, const float* logp_rollout, const float* adv,
                                      const uint8_t* mask, int64_t T, float eps_low, float eps_high,
                                      const int64_t* n_tokens, double* loss, float* g, uint8_t* flags,
                                      int64_t* counts, hipStream_t stream) {
  if (!logp || !logp_rollout || !adv || !mask || !loss || !g || !flags || !counts)
    return fail(SAO_ERR_NULL, "logp, logp_rollout, adv, mask, loss, g, flags and counts are required");
  if (T < 0 || T > kMaxRows) return fail(SAO_ERR_SHAPE, "T=%lld out of range", (long long)T);
  if (!(eps_low >= 0.0f) || !std::isfinite(eps_low) || !(eps_high >= 0.0f) || !std::isfinite(eps_high))
    return fail(SAO_ERR_VALUE, "eps_low=%g, eps_high=%g must be finite and >= 0", eps_low, eps_high);
  if (T == 0) return ok();
  const size_t need = sao::loss_layout(T).total;
  if (need > sao::kLossScratchBytes)
    return fail(SAO_ERR_WORKSPACE, "T=%lld needs %zu bytes of scratch, more than the static %zu", (long long)T,
                need, sao::kLossScratchBytes);
  return device(sao::launch_loss_noalloc(logp, logp_rollout, adv, mask, T, eps_low, eps_high, n_tokens, loss, g,
                                         flags, counts, stream),
                "sao_clipped_loss_noalloc launch");
}

sao_status_t sao_ppo_loss(const float* logp, const float* logp_old, const float* logp_behav, const float* adv,
                          const uint8_t* mask, int64_t T, float eps_low, float eps_high, const int64_t* n_tokens,
                          double* loss, float* g, uint8_t* flags, int64_t* counts, void* ws, size_t ws_bytes,
                          hipStream_t stream) {
  if (!logp || !logp_old || !adv || !mask || !loss || !g || !flags || !counts)
    return fail(SAO_ERR_NULL, "logp, logp_old, adv, mask, loss, g, flags and counts are required");
  if (T < 0 || T > kMaxRows) return fail(SAO_ERR_SHAPE, "T=%lld out of range", (long long)T);
  if (!(eps_low >= 0.0f) || !std::isfinite(eps_low) || !(eps_high >= 0.0f) || !std::isfinite(eps_high))
    return fail(SAO_ERR_VALUE, "eps_low=%g, eps_high=%g must be finite and >= 0", eps_low, eps_high);
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_PPO_LOSS, T, 1, 1, SAO_F32))) return s;
  return device(sao::launch_ppo_loss(logp, logp_old, logp_behav, adv, mask, T, eps_low, eps_high, n_tokens, loss,
                                     g, flags, counts, ws, stream),
                "sao_ppo_loss launch");
}

sao_status_t sao_explained_variance(const float* values, const float* ret, const uint8_t* mask, int64_t T,
                                    double* moments, double* ev, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (!values || !ret || !mask || !moments) return fail(SAO_ERR_NULL, "values, ret, mask and moments are required");
  if (T < 0 || T > kMaxRows) return fail(SAO_ERR_SHAPE, "T=%lld out of range", (long long)T);
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_EXPLAINED_VARIANCE, T, 1, 1, SAO_F32)))
    return s;
  return device(sao::launch_explained_variance(values, ret, mask, T, moments, ev, ws, stream),
                "sao_explained_variance launch");
}

sao_status_t sao_loss_backward(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w,
                               const int32_t* target, const float* lse, const float* g, int64_t T, int64_t H,
                               int64_t V, sao_dtype_t dtype, void* dhidden, float* dw_head, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  if (!hidden || !w_head || !target || !lse || !g || !dhidden || !dw_head)
    return fail(SAO_ERR_NULL, "hidden, w_head, target, lse, g, dhidden and dw_head are required");
  if (sao_status_t s = check_head(hidden, ld_hidden, w_head, ld_w, T, H, V, dtype)) return s;
  if (!aligned16(dhidden) || !aligned16(dw_head))
    return fail(SAO_ERR_SHAPE, "dhidden and dw_head must be 16-byte aligned");
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_BACKWARD, T, H, V, dtype))) return s;
  return device(sao::launch_backward(hidden, ld_hidden, w_head, ld_w, target, lse, g, T, H, V,
                                     dtype == SAO_BF16, dhidden, dw_head, ws, stream),
                "sao_loss_backward launch");
}

sao_status_t sao_value_forward(const void* hidden, int64_t ld_hidden, const void* w_v, int64_t T, int64_t H,
                               sao_dtype_t dtype, float* v, void* ws, size_t ws_bytes, hipStream_t stream) {
  (void)ws;
  (void)ws_bytes;
  if (!hidden || !w_v || !v) return fail(SAO_ERR_NULL, "hidden, w_v and v are required");
  if (sao_status_t s = check_head(hidden, ld_hidden, w_v, H, T, H, 1, dtype)) return s;
  if (T == 0) return ok();
  return device(sao::launch_value_forward(hidden, ld_hidden, w_v, T, H, dtype == SAO_BF16, v, stream),
                "sao_value_forward launch");
}

sao_status_t sao_value_loss(const void* hidden, int64_t ld_hidden, const void* w_v, const float* v,
                            const float* ret, const uint8_t* mask, int64_t T, int64_t H, const int64_t* n_tokens,
                            sao_dtype_t dtype, double* loss_v, void* dhidden_v, float* dw_v, void* ws,
                            size_t ws_bytes, hipStream_t stream) {
  if (!hidden || !w_v || !v || !ret || !mask || !loss_v || !dhidden_v || !dw_v)
    return fail(SAO_ERR_NULL, "hidden, w_v, v, ret, mask, loss_v, dhidden_v and dw_v are required");
  if (sao_status_t s = check_head(hidden, ld_hidden, w_v, H, T, H, 1, dtype)) return s;
  if (!aligned16(dhidden_v)) return fail(SAO_ERR_SHAPE, "dhidden_v must be 16-byte aligned");
  if (T == 0) return ok();
  if (sao_status_t s = check_ws(ws, ws_bytes, sao_workspace_size(SAO_OP_VALUE, T, H, 1, dtype))) return s;
  return device(sao::launch_value_loss(hidden, ld_hidden, w_v, v, ret, mask, T, H, n_tokens, dtype == SAO_BF16,
                                       loss_v, dhidden_v, dw_v, ws, stream),
                "sao_value_loss launch");
}

}  // extern "C"

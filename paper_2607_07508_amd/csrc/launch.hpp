// Internal launch entry points behind the C ABI (device pointers, caller's stream).
// Each returns the HIP status of its launches (0 on success) as an int, so that the
// argument-validation layer that calls them needs no HIP header.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/sao.h"

namespace sao {

int launch_logprob(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w,
                          const int32_t* target, const uint8_t* mask, int64_t T, int64_t H, int64_t V,
                          bool bf16, float* logp, float* lse, int32_t* status, void* ws, hipStream_t st);

int launch_backward(const void* hidden, int64_t ld_hidden, const void* w_head, int64_t ld_w,
                           const int32_t* target, const float* lse, const float* g, int64_t T, int64_t H,
                           int64_t V, bool bf16, void* dhidden, float* dw, void* ws, hipStream_t st);

int launch_advantage(const float* values, const float* rewards, const uint8_t* mask,
                            const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma, double lam,
                            double alpha, float* adv, float* ret, int64_t* n_tokens, int32_t* status,
                            void* ws, hipStream_t st);

int launch_step_advantage(const float* values, const float* rewards, const uint8_t* mask,
                                 const int32_t* cu_seqlens, int32_t B, int64_t T, double gamma, double lam,
                                 double alpha, bool last_value, float* adv, float* ret, uint8_t* last,
                                 int64_t* n_tokens, int32_t* status, void* ws, hipStream_t st);

int launch_group_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens, int32_t B,
                                  int64_t T, int32_t group_size, double eps_stab, float* adv, double* traj_reward,
                                  double* traj_adv, int64_t* n_tokens, int32_t* status, void* ws, hipStream_t st);

int launch_running_mean_advantage(const float* rewards, const uint8_t* mask, const int32_t* cu_seqlens,
                                         int32_t B, int64_t T, const int32_t* keys, int32_t n_keys, int32_t window,
                                         double* history, int64_t* seen, float* adv, double* traj_reward,
                                         double* traj_adv, int64_t* n_tokens, int32_t* status, void* ws,
                                         hipStream_t st);

int launch_loss(const float* logp, const float* logp_rollout, const float* adv, const uint8_t* mask,
                       int64_t T, float eps_low, float eps_high, const int64_t* n_tokens, double* loss,
                       float* g, uint8_t* flags, int64_t* counts, void* ws, hipStream_t st);

// The DIS loss with its workspace in a static per-device array of
// kLossScratchBytes (no allocation); the stream must belong to the current device.
int launch_loss_noalloc(const float* logp, const float* logp_rollout, const float* adv, const uint8_t* mask,
                        int64_t T, float eps_low, float eps_high, const int64_t* n_tokens, double* loss, float* g,
                        uint8_t* flags, int64_t* counts, hipStream_t st);

int launch_ppo_loss(const float* logp, const float* logp_old, const float* logp_behav, const float* adv,
                           const uint8_t* mask, int64_t T, float eps_low, float eps_high, const int64_t* n_tokens,
                           double* loss, float* g, uint8_t* flags, int64_t* counts, void* ws, hipStream_t st);

int launch_explained_variance(const float* values, const float* ret, const uint8_t* mask, int64_t T,
                                     double* moments, double* ev, void* ws, hipStream_t st);

int launch_value_forward(const void* hidden, int64_t ld_hidden, const void* w_v, int64_t T, int64_t H,
                                bool bf16, float* v, hipStream_t st);

int launch_value_loss(const void* hidden, int64_t ld_hidden, const void* w_v, const float* v,
                             const float* ret, const uint8_t* mask, int64_t T, int64_t H, const int64_t* n_tokens,
                             bool bf16, double* loss_v, void* dhidden_v, float* dw_v, void* ws, hipStream_t st);

// Text of a HIP status code returned by the launchers.
const char* device_error_string(int code);

}  // namespace sao

// Host-only stand-ins for the device side of the C ABI. Linked with api.cpp (and
// never into libsao.so) they give a library that validates arguments exactly as
// the real one does but has no GPU code, so that the validation layer can be
// built with a plain host compiler under the address and undefined-behaviour
// sanitizers. Every launcher reports a device error without touching its
// arguments; the measurement hook does nothing.
#include "../../include/sao.h"
#include "launch.hpp"

namespace sao {

namespace {
constexpr int kNoDevice = 100;  // any nonzero status reads as a device error
}

const char* device_error_string(int) { return "host-only build of the validation layer: no device"; }

int launch_logprob(const void*, int64_t, const void*, int64_t, const int32_t*, const uint8_t*, int64_t, int64_t,
                   int64_t, bool, float*, float*, int32_t*, void*, hipStream_t) {
  return kNoDevice;
}
int launch_backward(const void*, int64_t, const void*, int64_t, const int32_t*, const float*, const float*, int64_t,
                    int64_t, int64_t, bool, void*, float*, void*, hipStream_t) {
  return kNoDevice;
}
int launch_advantage(const float*, const float*, const uint8_t*, const int32_t*, int32_t, int64_t, double, double,
                     double, float*, float*, int64_t*, int32_t*, void*, hipStream_t) {
  return kNoDevice;
}
int launch_step_advantage(const float*, const float*, const uint8_t*, const int32_t*, int32_t, int64_t, double,
                          double, double, bool, float*, float*, uint8_t*, int64_t*, int32_t*, void*, hipStream_t) {
  return kNoDevice;
}
int launch_group_advantage(const float*, const uint8_t*, const int32_t*, int32_t, int64_t, int32_t, double, float*,
                           double*, double*, int64_t*, int32_t*, void*, hipStream_t) {
  return kNoDevice;
}
int launch_running_mean_advantage(const float*, const uint8_t*, const int32_t*, int32_t, int64_t, const int32_t*,
                                  int32_t, int32_t, double*, int64_t*, float*, double*, double*, int64_t*, int32_t*,
                                  void*, hipStream_t) {
  return kNoDevice;
}
int launch_loss(const float*, const float*, const float*, const uint8_t*, int64_t, float, float, const int64_t*,
                double*, float*, uint8_t*, int64_t*, void*, hipStream_t) {
  return kNoDevice;
}
int launch_loss_noalloc(const float*, const float*, const float*, const uint8_t*, int64_t, float, float,
                        const int64_t*, double*, float*, uint8_t*, int64_t*, hipStream_t) {
  return kNoDevice;
}
int launch_ppo_loss(const float*, const float*, const float*, const float*, const uint8_t*, int64_t, float, float,
                    const int64_t*, double*, float*, uint8_t*, int64_t*, void*, hipStream_t) {
  return kNoDevice;
}
int launch_explained_variance(const float*, const float*, const uint8_t*, int64_t, double*, double*, void*,
                              hipStream_t) {
  return kNoDevice;
}
int launch_value_forward(const void*, int64_t, const void*, int64_t, int64_t, bool, float*, hipStream_t) {
  return kNoDevice;
}
int launch_value_loss(const void*, int64_t, const void*, const float*, const float*, const uint8_t*, int64_t,
                      int64_t, const int64_t*, bool, double*, void*, float*, void*, hipStream_t) {
  return kNoDevice;
}

}  // namespace sao

extern "C" void sao_debug_time_kernel(int, void*, void*) {}
extern "C" void sao_debug_clock_samples(int, void*, int64_t) {}

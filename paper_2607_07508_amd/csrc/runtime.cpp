// The HIP side of the C ABI that is not a kernel launcher: text of HIP status
// codes, and the per-thread measurement hook.
#include <hip/hip_runtime.h>

#include "../../include/sao.h"
#include "launch.hpp"
#include "timer.hpp"

namespace sao {

const char* device_error_string(int code) { return hipGetErrorString(static_cast<hipError_t>(code)); }

KernelTimer& kernel_timer() {
  thread_local KernelTimer t;
  return t;
}

}  // namespace sao

extern "C" void sao_debug_clock_samples(int kernel, void* records, int64_t slots) {
  sao::KernelTimer& t = sao::kernel_timer();
  t.clocks = (kernel != SAO_KERNEL_NONE && records && slots > 0) ? static_cast<int64_t*>(records) : nullptr;
  t.clock_slots = t.clocks ? slots : 0;
  t.clock_kernel = t.clocks ? kernel : SAO_KERNEL_NONE;
}

extern "C" void sao_debug_time_kernel(int kernel, void* start_event, void* stop_event) {
  sao::KernelTimer& t = sao::kernel_timer();
  t.kernel = (start_event && stop_event) ? kernel : SAO_KERNEL_NONE;
  t.start = static_cast<hipEvent_t>(start_event);
  t.stop = static_cast<hipEvent_t>(stop_event);
}

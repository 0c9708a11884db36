// Per-thread measurement hook of sao_debug_time_kernel: the caller's event pair
// and the kernel it brackets.
#pragma once

#include <hip/hip_runtime.h>

namespace sao {

struct KernelTimer {
  int kernel = 0;
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
  int64_t* clocks = nullptr;  // per-workgroup clock records of the head forward (device), or null
  int64_t clock_slots = 0;    // records the buffer holds
};

// The calling thread's hook (thread-local state, the library's only mutable host state).
KernelTimer& kernel_timer();

}  // namespace sao

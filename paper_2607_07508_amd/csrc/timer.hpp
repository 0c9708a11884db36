// Per-thread measurement hook of sao_debug_time_kernel: the caller's event pair
// and the kernel it brackets.
#pragma once

#include <hip/hip_runtime.h>

namespace sao {

struct KernelTimer {
  int kernel = 0;
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
  int64_t* clocks = nullptr;  // per-workgroup clock records (device), or null
  int64_t clock_slots = 0;    // records the buffer holds
  int clock_kernel = 0;       // the kernel that records them

  // The event pair and the clock records for a launch of kernel `k` (null when off).
  bool timed(int k) const { return kernel == k && start && stop; }
  int64_t* clocks_for(int k) const { return clock_kernel == k ? clocks : nullptr; }
};

// The calling thread's hook (thread-local state, the library's only mutable host state).
KernelTimer& kernel_timer();

}  // namespace sao

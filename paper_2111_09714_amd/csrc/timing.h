// Opt-in per-kernel timing with HIP events (benchmarking aid, internal header).
// When enabled through yoso_timing_enable(), every kernel launch of the library
// is bracketed by a pair of events recorded on the launch stream.
#pragma once

#include <hip/hip_runtime.h>

namespace yoso {

class KernelTimer {
   public:
    KernelTimer(const char *kernel, hipStream_t stream);
    ~KernelTimer();
    KernelTimer(const KernelTimer &) = delete;
    KernelTimer &operator=(const KernelTimer &) = delete;

   private:
    hipEvent_t stop_ = nullptr;
    hipStream_t stream_;
};

}  // namespace yoso

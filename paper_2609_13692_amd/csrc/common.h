// Host-side pieces shared by the library's source files: the calling
// thread's error text, HIP error checks, the per-launch event profiler and
// launch-size helpers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "mpt.h"

namespace mptlib {

// Sets the calling thread's error text (printf format); returns status.
int fail(int status, const char *fmt, ...);
void clear_error();
const char *error_text();

// While profiling is on (mpt_profile_begin), records HIP events on the
// caller's stream around one launch, under `name`, with `work` algorithmic
// units.
class LaunchScope {
  public:
    LaunchScope(const char *name, double work, hipStream_t s);
    ~LaunchScope();
    LaunchScope(const LaunchScope &) = delete;
    LaunchScope &operator=(const LaunchScope &) = delete;

  private:
    hipStream_t s_;
    bool active_ = false;
    hipEvent_t a_{}, b_{};
    const char *name_;
    double work_;
};

inline int grid_for(int64_t n, int threads, int cap = 8192) {
    int64_t g = (n + threads - 1) / threads;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

inline size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

}  // namespace mptlib

#define MPT_HIP_TRY(expr)                                                                  \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return mptlib::fail(MPT_E_DEVICE, "%s: %s (%s:%d)", #expr, hipGetErrorString(e_), \
                                __FILE__, __LINE__);                                       \
    } while (0)

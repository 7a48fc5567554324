// Host-side pieces shared by the library's source files: the calling
// thread's error text, HIP error checks, the per-launch event profiler,
// launch-size helpers and the exception guard of the exported calls.
#pragma once

#include <hip/hip_runtime.h>
#include <rocprofiler-sdk-roctx/roctx.h>

#include <cstddef>
#include <cstdint>
#include <exception>

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

// A named roctx range around one phase of an exported call (visible to
// rocprofv3 --marker-trace; a no-op without a profiler).
class Range {
  public:
    explicit Range(const char *name) { roctxRangePushA(name); }
    ~Range() { roctxRangePop(); }
    Range(const Range &) = delete;
    Range &operator=(const Range &) = delete;
};

inline int grid_for(int64_t n, int threads, int cap = 8192) {
    int64_t g = (n + threads - 1) / threads;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

inline size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// Runs the body of an exported call: a C++ exception never crosses the C ABI,
// it becomes MPT_E_INTERNAL with its text.
template <class F>
inline int guarded(const char *where, F &&body) noexcept {
    try {
        return body();
    } catch (const std::exception &e) {
        return fail(MPT_E_INTERNAL, "%s: %s", where, e.what());
    } catch (...) {
        return fail(MPT_E_INTERNAL, "%s: unexpected exception", where);
    }
}

}  // namespace mptlib

#define MPT_HIP_TRY(expr)                                                                  \
    do {                                                                                   \
        hipError_t e_ = (expr);                                                            \
        if (e_ != hipSuccess)                                                              \
            return mptlib::fail(MPT_E_DEVICE, "%s: %s (%s:%d)", #expr, hipGetErrorString(e_), \
                                __FILE__, __LINE__);                                       \
    } while (0)

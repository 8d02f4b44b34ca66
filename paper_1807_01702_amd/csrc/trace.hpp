// trace.hpp -- optional per-launch timing of the library's kernels (the
// bnr_trace_begin / bnr_trace_end diagnostics).  When a launch's class is
// selected, two HIP events are recorded on the launch stream around it and
// the launch's algorithmic HBM bytes and floating-point operations are kept
// with them.
#pragma once
#include <hip/hip_runtime.h>

namespace bnr {

enum KernelClass { KC_CONV = 1, KC_WGRAD = 2, KC_SWEEP = 4, KC_SMALL = 8 };
enum KernelId {
    KID_CONV_1X1 = 1, KID_CONV_3X3 = 2, KID_WGRAD_1X1 = 3, KID_WGRAD_3X3 = 4, KID_STATS_SWEEP = 5,
    KID_ELEMENTWISE = 6, KID_COMBINE = 7, KID_PACK = 8, KID_SPLITK_SUM = 9, KID_POOL = 10, KID_COPY = 11,
    KID_STEM_CONV = 12, KID_STEM_WGRAD = 13, KID_MAXPOOL = 14, KID_HEAD = 15
};

bool trace_wants(int kernel_class);
void trace_record(hipEvent_t a, hipEvent_t b, double bytes, double flops, int kid);

// While one of these lives on a thread, that thread's launches are not traced
// (no events are created): the entry point that allocates nothing uses it.
struct TraceSuppress {
    TraceSuppress();
    ~TraceSuppress();
};

// RAII bracket around one launch (no-op unless tracing selects its class)
class TraceScope {
  public:
    TraceScope(int cls, int kid, hipStream_t s, double bytes, double flops)
        : on_(trace_wants(cls)), s_(s), bytes_(bytes), flops_(flops), kid_(kid) {
        if (on_ && hipEventCreate(&a_) == hipSuccess && hipEventCreate(&b_) == hipSuccess) {
            on_ = hipEventRecord(a_, s_) == hipSuccess;
        } else {
            on_ = false;
        }
    }
    ~TraceScope() {
        if (on_ && hipEventRecord(b_, s_) == hipSuccess) trace_record(a_, b_, bytes_, flops_, kid_);
    }
  private:
    bool on_;
    hipStream_t s_;
    hipEvent_t a_ = nullptr, b_ = nullptr;
    double bytes_, flops_;
    int kid_;
};

}  // namespace bnr

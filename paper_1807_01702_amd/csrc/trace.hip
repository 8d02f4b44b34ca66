// trace.hip -- state of the launch-timing diagnostics (bnr_trace_begin/end).
#include <atomic>
#include <mutex>
#include <vector>

#include "../../include/bnr.h"
#include "trace.hpp"

namespace bnr {
namespace {
struct Rec { hipEvent_t a, b; double bytes, flops; int kid; };
std::mutex g_mu;                       // guards g_cap and g_recs
std::atomic<int> g_classes{0};         // selected classes; 0 = tracing off
size_t g_cap = 0;
std::vector<Rec> g_recs;
thread_local int g_suppress = 0;
}  // namespace

TraceSuppress::TraceSuppress() { g_suppress++; }
TraceSuppress::~TraceSuppress() { g_suppress--; }

// Tracing off (the normal case) costs one relaxed load per launch, no lock.
bool trace_wants(int kernel_class)
{
    if (g_suppress || (g_classes.load(std::memory_order_relaxed) & kernel_class) == 0) return false;
    std::lock_guard<std::mutex> lk(g_mu);
    return (g_classes.load(std::memory_order_relaxed) & kernel_class) != 0 && g_recs.size() < g_cap;
}

void trace_record(hipEvent_t a, hipEvent_t b, double bytes, double flops, int kid)
{
    std::lock_guard<std::mutex> lk(g_mu);
    g_recs.push_back(Rec{a, b, bytes, flops, kid});
}

}  // namespace bnr

extern "C" {

bnr_status bnr_trace_begin(int32_t kernel_classes, int32_t capacity)
{
    if (capacity <= 0 || kernel_classes <= 0) return BNR_ERR_SHAPE;
    std::lock_guard<std::mutex> lk(bnr::g_mu);
    for (auto &r : bnr::g_recs) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
    bnr::g_recs.clear();
    bnr::g_recs.reserve((size_t)capacity);
    bnr::g_cap = (size_t)capacity;
    bnr::g_classes.store(kernel_classes, std::memory_order_relaxed);
    return BNR_OK;
}

int32_t bnr_trace_end(double *ms, double *bytes, double *flops, int32_t *kernel_id, int32_t capacity)
{
    std::vector<bnr::Rec> recs;
    {
        std::lock_guard<std::mutex> lk(bnr::g_mu);
        recs.swap(bnr::g_recs);
        bnr::g_classes.store(0, std::memory_order_relaxed);
        bnr::g_cap = 0;
    }
    int32_t n = 0;
    for (auto &r : recs) {
        if (n < capacity) {
            float t = 0.f;
            if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&t, r.a, r.b) != hipSuccess) t = -1.f;
            if (ms) ms[n] = t;
            if (bytes) bytes[n] = r.bytes;
            if (flops) flops[n] = r.flops;
            if (kernel_id) kernel_id[n] = r.kid;
            n++;
        }
        (void)hipEventDestroy(r.a);
        (void)hipEventDestroy(r.b);
    }
    return n;
}

}  // extern "C"

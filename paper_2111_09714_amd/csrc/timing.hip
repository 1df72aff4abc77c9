// Opt-in per-kernel timing with HIP events (host code only).
//
// Disabled by default: then a KernelTimer costs one relaxed atomic load.  When
// enabled, each kernel name owns a pool of `capacity` event pairs created on its
// first launch; launches beyond the pool are not recorded.  Queries synchronise
// on the recorded events and sum their elapsed times.
#include <atomic>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/yoso.h"
#include "timing.h"

namespace yoso {

namespace {

struct Pool {
    std::vector<hipEvent_t> start, stop;
    size_t used = 0;
};

std::atomic<bool> g_enabled{false};
std::mutex g_mu;
std::map<std::string, Pool> g_pools;
size_t g_capacity = 0;

void destroy_all() {
    for (auto &kv : g_pools) {
        for (hipEvent_t e : kv.second.start) (void)hipEventDestroy(e);
        for (hipEvent_t e : kv.second.stop) (void)hipEventDestroy(e);
    }
    g_pools.clear();
}

}  // namespace

KernelTimer::KernelTimer(const char *kernel, hipStream_t stream) : stream_(stream) {
    if (!g_enabled.load(std::memory_order_relaxed)) return;
    std::lock_guard<std::mutex> lock(g_mu);
    Pool &p = g_pools[kernel];
    if (p.start.empty()) {
        p.start.resize(g_capacity, nullptr);
        p.stop.resize(g_capacity, nullptr);
        for (size_t i = 0; i < g_capacity; i++) {
            if (hipEventCreate(&p.start[i]) != hipSuccess || hipEventCreate(&p.stop[i]) != hipSuccess) {
                p.start.resize(i);
                p.stop.resize(i);
                break;
            }
        }
    }
    if (p.used >= p.start.size()) return;
    (void)hipEventRecord(p.start[p.used], stream_);
    stop_ = p.stop[p.used];
    p.used++;
}

KernelTimer::~KernelTimer() {
    if (stop_) (void)hipEventRecord(stop_, stream_);
}

}  // namespace yoso

extern "C" {

yoso_status yoso_timing_enable(int32_t capacity) {
    std::lock_guard<std::mutex> lock(yoso::g_mu);
    yoso::destroy_all();
    yoso::g_capacity = capacity > 0 ? (size_t)capacity : 0;
    yoso::g_enabled.store(capacity > 0);
    return YOSO_OK;
}

yoso_status yoso_timing_reset(void) {
    std::lock_guard<std::mutex> lock(yoso::g_mu);
    for (auto &kv : yoso::g_pools) kv.second.used = 0;
    return YOSO_OK;
}

yoso_status yoso_timing_query(const char *kernel, double *total_ms, int64_t *launches) {
    if (kernel == nullptr || total_ms == nullptr || launches == nullptr) return YOSO_ERR_NULL;
    std::lock_guard<std::mutex> lock(yoso::g_mu);
    *total_ms = 0.0;
    *launches = 0;
    auto it = yoso::g_pools.find(kernel);
    if (it == yoso::g_pools.end()) return YOSO_OK;
    const yoso::Pool &p = it->second;
    for (size_t i = 0; i < p.used; i++) {
        if (hipEventSynchronize(p.stop[i]) != hipSuccess) return YOSO_ERR_DEVICE;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, p.start[i], p.stop[i]) != hipSuccess) return YOSO_ERR_DEVICE;
        *total_ms += ms;
    }
    *launches = (int64_t)p.used;
    return YOSO_OK;
}

}  // extern "C"

// Kernel timing for diagnostics: HIP event pairs around launches of armed
// kernel kinds, recorded on the launch stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "device.h"

namespace ms {

namespace {
constexpr int kKinds = 6;
constexpr size_t kMaxLaunches = 65536;

struct KindLog {
    std::vector<hipEvent_t> begin, end;   // one pair per recorded launch
};

std::mutex g_mu;
unsigned g_armed = 0;
KindLog g_log[kKinds];
std::vector<hipEvent_t> g_pool;           // events reusable across sessions
bool g_open[kKinds] = {false, false, false, false, false, false};

int kind_index(unsigned kind) {
    for (int i = 0; i < kKinds; ++i)
        if (kind == (1u << i)) return i;
    return -1;
}

hipEvent_t take_event() {
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    // timing only: no system-scope fence (cache writeback and invalidate)
    // when the event completes, so the pair measures the kernel and not the
    // fence, and the following work is not slowed by it
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

void recycle(KindLog &l) {
    for (hipEvent_t e : l.begin) g_pool.push_back(e);
    for (hipEvent_t e : l.end) g_pool.push_back(e);
    l.begin.clear();
    l.end.clear();
}
}  // namespace

namespace {
thread_local bool t_off = false;
}  // namespace

void prof_thread_off(bool off) { t_off = off; }

void prof_mark(unsigned kind, void *stream, bool begin) {
    if (t_off || !(g_armed & kind)) return;   // unarmed fast path (racy read is harmless)
    std::lock_guard<std::mutex> lk(g_mu);
    if (!(g_armed & kind)) return;
    const int k = kind_index(kind);
    if (k < 0) return;
    KindLog &l = g_log[k];
    if (begin) {
        if (l.begin.size() >= kMaxLaunches) return;
        hipEvent_t e = take_event();
        if (!e) return;
        (void)hipEventRecord(e, (hipStream_t)stream);
        l.begin.push_back(e);
        g_open[k] = true;
    } else {
        if (!g_open[k]) return;
        hipEvent_t e = take_event();
        if (!e) {
            g_pool.push_back(l.begin.back());
            l.begin.pop_back();
        } else {
            (void)hipEventRecord(e, (hipStream_t)stream);
            l.end.push_back(e);
        }
        g_open[k] = false;
    }
}

bool prof_pair(unsigned kind, void **begin, void **end) {
    *begin = *end = nullptr;
    if (t_off || !(g_armed & kind)) return false;
    std::lock_guard<std::mutex> lk(g_mu);
    const int k = kind_index(kind);
    if (k < 0 || !(g_armed & kind) || g_log[k].begin.size() >= kMaxLaunches) return false;
    hipEvent_t b = take_event();
    if (!b) return false;
    hipEvent_t e = take_event();
    if (!e) {
        g_pool.push_back(b);
        return false;
    }
    *begin = b;
    *end = e;
    return true;
}

void prof_pair_done(unsigned kind, void *begin, void *end, bool launched) {
    std::lock_guard<std::mutex> lk(g_mu);
    const int k = kind_index(kind);
    if (k >= 0 && launched && (g_armed & kind)) {
        g_log[k].begin.push_back((hipEvent_t)begin);
        g_log[k].end.push_back((hipEvent_t)end);
    } else {
        g_pool.push_back((hipEvent_t)begin);
        g_pool.push_back((hipEvent_t)end);
    }
}

int prof_start(unsigned kinds) {
    std::lock_guard<std::mutex> lk(g_mu);
    for (int i = 0; i < kKinds; ++i) {
        // events of the previous session may still be pending on a stream
        for (hipEvent_t e : g_log[i].end) (void)hipEventSynchronize(e);
        recycle(g_log[i]);
        g_open[i] = false;
    }
    g_armed = kinds;
    return 0;
}

int prof_read(unsigned kind, uint64_t *launches, double *total_ms) {
    std::lock_guard<std::mutex> lk(g_mu);
    const int k = kind_index(kind);
    *launches = 0;
    *total_ms = 0.0;
    if (k < 0) return (int)hipErrorInvalidValue;
    KindLog &l = g_log[k];
    const size_t n = std::min(l.begin.size(), l.end.size());
    double tot = 0.0;
    for (size_t i = 0; i < n; ++i) {
        hipError_t e = hipEventSynchronize(l.end[i]);
        if (e != hipSuccess) return (int)e;
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, l.begin[i], l.end[i]);
        if (e != hipSuccess) return (int)e;
        tot += ms;
    }
    *launches = n;
    *total_ms = tot;
    return 0;
}

}  // namespace ms

// Per-(device, stream) transient workspace for split-K partials and
// reduction partials.  A buffer is reused by every call on its stream (the
// stream orders those calls); it only grows, and growth first waits for the
// stream so the old buffer is no longer in use.
//
// Also the fixed scratch array of the no-allocation backward: a file-scope
// device array that every GPU the library runs on holds from the first
// kernel launch until the process ends.  Host code never uses the array's
// name as an address (on the host it is only a stand-in for the symbol);
// its device address is looked up once per device with
// hipGetSymbolAddress and kept.
#include <hip/hip_runtime.h>

#include <atomic>
#include <map>
#include <mutex>
#include <utility>

#include "device.h"

namespace ms {

namespace {
struct Buf {
    void *p = nullptr;
    size_t n = 0;
};
std::mutex g_mu;
std::map<std::pair<int, void *>, Buf> g_bufs;
std::atomic<int> g_fail_next{0};
}  // namespace

void workspace_fail_next(int n) { g_fail_next.store(n); }

// err: 0 ok, 1 allocation failed, 2 other HIP error
void *workspace_get(void *stream, size_t bytes, int *err) {
    *err = 0;
    if (bytes == 0) return nullptr;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) {
        *err = 2;
        return nullptr;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    Buf &b = g_bufs[{dev, stream}];
    if (b.n >= bytes) return b.p;
    if (g_fail_next.load() > 0) {
        g_fail_next.fetch_sub(1);
        *err = 1;
        return nullptr;
    }
    if (b.p) {
        if (hipStreamSynchronize((hipStream_t)stream) != hipSuccess) {
            *err = 2;
            return nullptr;
        }
        (void)hipFree(b.p);
        b.p = nullptr;
        b.n = 0;
    }
    const size_t gran = size_t(2) << 20;
    const size_t want = (bytes + gran - 1) / gran * gran;
    if (hipMalloc(&b.p, want) != hipSuccess) {
        (void)hipGetLastError();
        b.p = nullptr;
        *err = 1;
        return nullptr;
    }
    b.n = want;
    return b.p;
}

int device_last_error() { return (int)hipGetLastError(); }

// ------------------------------------------------------------------ fixed scratch
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

// err: 0 ok, 1 the request exceeds kScratchBytes, 2 HIP error (no device, or
// the symbol lookup failed)
void *scratch_get(size_t bytes, int *err) {
    *err = 0;
    if (bytes > kScratchBytes) {
        *err = 1;
        return nullptr;
    }
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
        *err = 2;
        return nullptr;
    }
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        // once per device, with that device current: each GPU holds its own
        // copy of the array at its own address
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            *err = 2;
            return nullptr;
        }
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

}  // namespace ms

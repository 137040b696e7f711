// Stub kernel launchers for host-only tests of the runtime (memsave.cpp).
//
// Linked in place of the HIP launchers, they launch nothing: each checks
// that every pointer the real kernel would dereference for the requested
// outputs is non-null and 16-byte-or-better plausible, logs the call, and
// returns 0 -- or 77 when the host runtime handed a kernel a pointer it
// must not use.  The workspace comes from host memory that nobody touches.
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../paper_2404_12406_amd/csrc/device.h"

namespace {
std::mutex g_mu;
std::string g_log;
std::string g_violation;
int g_fail_next = 0;
std::vector<void *> g_ws;
struct Freer {
    ~Freer() {
        for (void *p : g_ws) std::free(p);
    }
} g_freer;

void log(const char *s) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_log += s;
    g_log += ';';
}

int need(bool ok, const char *what) {
    if (ok) return 0;
    std::lock_guard<std::mutex> lk(g_mu);
    g_violation += what;
    g_violation += ';';
    return 77;
}
}  // namespace

extern "C" {
const char *stub_log() { return g_log.c_str(); }
const char *stub_violations() { return g_violation.c_str(); }
void stub_reset() {
    std::lock_guard<std::mutex> lk(g_mu);
    g_log.clear();
    g_violation.clear();
}
// workspace growths (allocations) since the library was loaded
long stub_workspace_allocations() {
    std::lock_guard<std::mutex> lk(g_mu);
    return (long)g_ws.size();
}
}

namespace ms {

size_t conv_fwd_workspace(int, const ConvGeom &g) { return g.C % 8 ? 256 : 0; }

int launch_conv_fwd(int, const ConvGeom &g, const void *x, const void *w, const void *, void *y, void *ws, void *) {
    log("conv_fwd");
    if (g.C % 8 && (long long)g.N * g.P * g.Q * g.K > 0) need(ws, "conv_fwd:ws");
    const long long out = (long long)g.N * g.P * g.Q * g.K;
    const long long red = (long long)g.R * g.S * g.C;
    int e = 0;
    if (out > 0) e |= need(y, "conv_fwd:y");
    if (out > 0 && red > 0) e |= need(x && w, "conv_fwd:x,w");
    return e;
}

size_t conv_dgrad_workspace(int dtype, const ConvGeom &g, bool) {
    return dtype == kBF16 ? (size_t)g.K * g.R * g.S * g.C * 2 : 0;
}

// never takes the bias gradient along: the runtime then launches the column sum
int launch_conv_dgrad(int dtype, const ConvGeom &g, const void *dy, const void *w, const void *bias, void *dx,
                      void *ws, void *, void *, bool *db_done) {
    if (db_done) *db_done = false;
    log(bias ? "conv_dgrad+bias" : "conv_dgrad");
    if (conv_dgrad_workspace(dtype, g) > 0 && !ws) return need(false, "conv_dgrad:ws");
    const long long out = (long long)g.N * g.H * g.W * g.C;
    int e = 0;
    if (out > 0) e |= need(dx && w, "conv_dgrad:dx,w");
    if (out > 0 && (long long)g.N * g.P * g.Q * g.K > 0) e |= need(dy, "conv_dgrad:dy");
    return e;
}

size_t conv_wgrad_workspace(int, const ConvGeom &g, bool with_db) {
    const long long red = (long long)g.N * g.P * g.Q;
    return (red > 4096 ? (size_t)4 * g.K * g.R * g.S * g.C * 4 : 0) + (with_db ? (size_t)4 * g.K * 4 : 0);
}

// Like the bf16 fast path, fuses the bias gradient when asked for it (the
// fp32 path does not: the host must then launch the column sum itself).
int launch_conv_wgrad(int dtype, const ConvGeom &g, const void *dy, const void *x, void *dw, void *db, void *ws,
                      void *, bool *db_done) {
    log(db && dtype == kBF16 ? "conv_wgrad+db" : "conv_wgrad");
    *db_done = db != nullptr && dtype == kBF16;
    int e = 0;
    if ((long long)g.K * g.R * g.S * g.C > 0) e |= need(dw, "conv_wgrad:dw");
    if ((long long)g.N * g.P * g.Q > 0) e |= need(dy && x, "conv_wgrad:dy,x");
    if (conv_wgrad_workspace(dtype, g, db != nullptr) > 0) e |= need(ws, "conv_wgrad:ws");
    return e;
}

size_t conv3d_fwd_workspace(int, const Conv3dGeom &q) { return (size_t)q.g.N * q.g.H * q.g.W * q.g.C * 2 + 256; }
size_t conv3d_dgrad_workspace(int, const Conv3dGeom &q) { return (size_t)q.g.N * q.g.H * q.g.W * q.g.C * 2 + 512; }
size_t conv3d_wgrad_workspace(int, const Conv3dGeom &q, bool) { return (size_t)q.g.N * q.g.H * q.g.W * q.g.C * 2 + 768; }

int launch_conv3d_fwd(int, const Conv3dGeom &q, const void *u, const void *w, const void *, void *v, void *ws,
                      void *) {
    log("conv3d_fwd");
    int e = need(ws, "conv3d_fwd:ws");
    if ((long long)q.g.N * q.g.P * q.g.Q * q.g.K > 0) e |= need(u && w && v, "conv3d_fwd:u,w,v");
    return e;
}

int launch_conv3d_dgrad(int, const Conv3dGeom &q, const void *dv, const void *w, const void *bias, void *du,
                        void *ws, void *) {
    log(bias ? "conv3d_dgrad+bias" : "conv3d_dgrad");
    int e = need(ws, "conv3d_dgrad:ws");
    if ((long long)q.N * q.Din * q.g.H * q.g.W * q.C > 0) e |= need(dv && w && du, "conv3d_dgrad:dv,w,du");
    return e;
}

int launch_conv3d_wgrad(int dtype, const Conv3dGeom &q, const void *dv, const void *u, void *dw, void *db, void *ws,
                        void *, bool *db_done) {
    log(db && dtype == kBF16 ? "conv3d_wgrad+db" : "conv3d_wgrad");
    *db_done = db != nullptr && dtype == kBF16;
    int e = need(ws && dw, "conv3d_wgrad:ws,dw");
    if ((long long)q.g.N * q.g.P * q.g.Q > 0) e |= need(dv && u, "conv3d_wgrad:dv,u");
    return e;
}

size_t colsum_workspace(int, int64_t, int cols) { return (size_t)cols * 4 * 8; }

int launch_colsum(int, const void *in, int64_t rows, int cols, void *out, void *ws, void *) {
    log("colsum");
    int e = 0;
    if (cols > 0) e |= need(out && ws, "colsum:out,ws");
    if (rows > 0 && cols > 0) e |= need(in, "colsum:in");
    return e;
}

int launch_bn_fwd(int, const void *x, const void *mean, const void *var, const void *, const void *, float,
                  int64_t rows, int C, void *y, void *) {
    log("bn_fwd");
    if (rows > 0 && C > 0) return need(x && y && mean && var, "bn_fwd:x,y,mean,var");
    return 0;
}

size_t bn_bwd_workspace(int, int64_t, int C) { return (size_t)C * 4 * 16; }

int launch_bn_bwd(int, const void *dy, const void *x, const void *mean, const void *var, const void *gamma,
                  float, int64_t rows, int C, void *dx, void *dgamma, void *dbeta, void *ws, void *) {
    (void)gamma;
    log("bn_bwd");
    int e = 0;
    if (rows > 0 && C > 0) e |= need(dy, "bn_bwd:dy");
    if (dx || dgamma) e |= need(var, "bn_bwd:var");
    if (dgamma) e |= need(x && mean, "bn_bwd:x,mean");
    if (dgamma || dbeta) e |= need(ws, "bn_bwd:ws");
    return e;
}

int launch_relu_fwd(int, const void *x, int64_t n, void *y, void *bits, int64_t bits_bytes, void *) {
    log(bits ? "relu_fwd+bits" : "relu_fwd");
    int e = 0;
    if (n > 0) e |= need(x && y, "relu_fwd:x,y");
    if (bits_bytes > 0) e |= need(bits, "relu_fwd:bits");
    return e;
}

int launch_dropout(int, const void *in, int64_t n, void *out, uint64_t, uint64_t, uint32_t, float, int drop_all,
                   void *) {
    log(drop_all ? "dropout(all)" : "dropout");
    if (n > 0) return need(in && out, "dropout:in,out");
    return 0;
}

int launch_relu_bwd(int, const void *dy, const void *bits, int64_t n, void *dx, void *) {
    log("relu_bwd");
    return n > 0 ? need(dy && bits && dx, "relu_bwd:dy,bits,dx") : 0;
}

int launch_avgpool_fwd(int, const void *x, int N, int, int C, void *y, void *) {
    log("avgpool_fwd");
    return (N > 0 && C > 0) ? need(x && y, "avgpool_fwd:x,y") : 0;
}

int launch_avgpool_bwd(int, const void *dy, int N, int L, int C, void *dx, void *) {
    log("avgpool_bwd");
    return (N > 0 && C > 0 && L > 0) ? need(dy && dx, "avgpool_bwd:dy,dx") : 0;
}

void *workspace_get(void *, size_t bytes, int *err) {
    *err = 0;
    if (bytes == 0) return nullptr;
    std::lock_guard<std::mutex> lk(g_mu);
    if (g_fail_next > 0) {
        --g_fail_next;
        *err = 1;
        return nullptr;
    }
    void *p = std::malloc(bytes);
    g_ws.push_back(p);
    return p;
}

void workspace_fail_next(int n) {
    std::lock_guard<std::mutex> lk(g_mu);
    g_fail_next = n;
}

int launch_bn_nchw(int, const void *x, const void *, const void *var, const void *, const void *, float, int64_t N,
                   int C, int64_t HW, void *y, void *, bool backward) {
    log(backward ? "bn_nchw_bwd" : "bn_nchw");
    return N * C * HW > 0 ? need(x && var && y, "bn_nchw:x,var,y") : 0;
}

int launch_copy4(int, const void *src, const int64_t ext[4], const int64_t *, void *dst, const int64_t *, void *) {
    log("copy4");
    const long long n = (long long)ext[0] * ext[1] * ext[2] * ext[3];
    return n > 0 ? need(src && dst, "copy4:src,dst") : 0;
}

// the stub launchers never dereference workspace: any distinct non-null
// address stands in for the fixed scratch array
void *scratch_get(size_t bytes, int *err) {
    static char stand_in[256];
    *err = bytes > kScratchBytes ? 1 : 0;
    if (*err) return nullptr;
    log("scratch");
    return stand_in;
}

int gemm_plan_info(int, const ConvGeom &, int out[10]) {
    for (int i = 0; i < 10; ++i) out[i] = 0;
    return -1;
}

int device_last_error() { return 0; }

void prof_mark(unsigned, void *, bool) {}
void prof_thread_off(bool) {}
int prof_start(unsigned) { return 0; }
int prof_read(unsigned, uint64_t *launches, double *total_ms) {
    *launches = 0;
    *total_ms = 0.0;
    return 0;
}

}  // namespace ms

// Interface between the host runtime (memsave.cpp, plain C++) and the HIP
// kernel launchers (kernels/*.hip).  Plain types only, so the host runtime
// compiles without HIP headers.  Every launcher enqueues on `stream` (a
// hipStream_t) and returns 0 or the hipError_t of the failed launch.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace ms {

enum Dtype : int { kF32 = 0, kBF16 = 1 };

// Convolution geometry.  Activations are NHWC, filters KRSC, all dense.
// The fully-connected layer is the special case H = W = R = S = P = Q = 1,
// stride 1, pad 0 (x[M,K_in] = NHWC with N = M, C = K_in; W[N_out,K_in] = KRSC).
struct ConvGeom {
    int N, C, H, W;   // input
    int K, R, S;      // filters
    int P, Q;         // output extent
    int sh, sw, ph, pw;
};

// y = W * x + b (b may be null).  May use conv_fwd_workspace() bytes of
// workspace (zero-padded channel copies when C is not a multiple of 8).
size_t conv_fwd_workspace(int dtype, const ConvGeom &g);
int launch_conv_fwd(int dtype, const ConvGeom &g, const void *x, const void *w,
                    const void *bias, void *y, void *ws, void *stream);

// dx = input gradient of the convolution for grad dy (needs w only), plus
// bias[c] per channel when bias is non-null (the forward of a transposed
// convolution is this contraction).  May use conv_dgrad_workspace() bytes of
// workspace (a transposed copy of w, zero-padded channel copies).  When db
// is non-null the launcher may also produce the bias gradient db[k] = sum
// over pixels of dy[.][k] (bf16 unit geometry: the contraction's blocks add
// dy's columns as they finish) and sets *db_done; with_db sizes the
// workspace for that.
size_t conv_dgrad_workspace(int dtype, const ConvGeom &g, bool with_db = false);
int launch_conv_dgrad(int dtype, const ConvGeom &g, const void *dy, const void *w,
                      const void *bias, void *dx, void *ws, void *stream, void *db = nullptr,
                      bool *db_done = nullptr);

// The bf16 GEMM planner's decision for one contraction of a convolution
// (testing and diagnostics; launches nothing): pass 0 forward, 1 input
// gradient, 2 weight gradient.  out[0..9] = tile rows, tile columns, waves,
// LDS stages, k-groups, splits, input gradient reading W in place (1) or its
// transposed copy (0), columns of the first launch of a column split (0:
// none), the second launch's tile rows and columns.  Returns 0, or -1 when
// the fast path does not take the contraction.
int gemm_plan_info(int pass, const ConvGeom &g, int out[10]);

// dw = weight gradient for grad dy and input x.  Needs conv_wgrad_workspace()
// bytes of device workspace (may be 0).  When db is non-null the launcher may
// also produce the bias gradient db[k] = sum over pixels of dy[.][k] from the
// operand tiles it already reads; *db_done tells whether it did.
size_t conv_wgrad_workspace(int dtype, const ConvGeom &g, bool with_db);
int launch_conv_wgrad(int dtype, const ConvGeom &g, const void *dy, const void *x,
                      void *dw, void *db, void *ws, void *stream, bool *db_done);

// 3-D convolution u[N][Din][H][W][C] -> v[N][Do][P][Q][K], filter
// W[K][T][R][S][C] (depth taps T, depth stride sd, depth pad pd), run as the
// 2-D convolution g over N*Do images of the depth-folded input
// [N*Do][H][W][T*C] with the filter regrouped to [K][R][S][T*C]
// (conv3d.hip).  g.N = N*Do, g.C = T*C; g's other fields are the 3-D
// convolution's (H, W, K, R, S, P, Q, strides and pads).
struct Conv3dGeom {
    ConvGeom g;
    int N, C, Din, Do, T, sd, pd;
};
// v = conv(u) + bias (bias may be null)
size_t conv3d_fwd_workspace(int dtype, const Conv3dGeom &q);
int launch_conv3d_fwd(int dtype, const Conv3dGeom &q, const void *u, const void *w, const void *bias, void *v,
                      void *ws, void *stream);
// du = input gradient for dv (+ bias[c] when non-null: the transposed layer's forward)
size_t conv3d_dgrad_workspace(int dtype, const Conv3dGeom &q);
int launch_conv3d_dgrad(int dtype, const Conv3dGeom &q, const void *dv, const void *w, const void *bias, void *du,
                        void *ws, void *stream);
// dw = weight gradient for dv and u; db as launch_conv_wgrad
size_t conv3d_wgrad_workspace(int dtype, const Conv3dGeom &q, bool with_db);
int launch_conv3d_wgrad(int dtype, const Conv3dGeom &q, const void *dv, const void *u, void *dw, void *db, void *ws,
                        void *stream, bool *db_done);

// out[j] = sum_i in[i][j] for a dense row-major [rows][cols] matrix (bias
// gradient of conv over N*P*Q rows, of linear over M rows).
size_t colsum_workspace(int dtype, int64_t rows, int cols);
// out[j] = sum_i part[i][j] over `rows` fp32 partial rows (fixed order),
// rounded once to dtype.
int launch_colsum_finalize(int dtype, const float *part, int rows, int cols, void *out, void *stream);
int launch_colsum(int dtype, const void *in, int64_t rows, int cols, void *out,
                  void *ws, void *stream);

// BN-eval over x[rows][C] (NHWC pixels x channels).  gamma/beta may be null,
// and so may mean (read as zeros: the input gradient dy * gamma / sqrt(var + eps)).
int launch_bn_fwd(int dtype, const void *x, const void *mean, const void *var,
                  const void *gamma, const void *beta, float eps, int64_t rows, int C,
                  void *y, void *stream);
// BN-eval over a plain row-major [N, C, H, W] tensor (HW = H * W), in the
// same layout: the forward, or (mean and beta null) a backward that wants dx
// alone, dx = dy * gamma / sqrt(var + eps).  `backward` picks the profiling
// kind the launch counts as.
int launch_bn_nchw(int dtype, const void *x, const void *mean, const void *var, const void *gamma, const void *beta,
                   float eps, int64_t N, int C, int64_t HW, void *y, void *stream, bool backward);
size_t bn_bwd_workspace(int dtype, int64_t rows, int C);
// Any of dx, dgamma, dbeta may be null (not requested); x and mean are read
// only when dgamma is requested.
int launch_bn_bwd(int dtype, const void *dy, const void *x, const void *mean,
                  const void *var, const void *gamma, float eps, int64_t rows, int C,
                  void *dx, void *dgamma, void *dbeta, void *ws, void *stream);

// ReLU over n elements in memory order: y = x < 0 ? 0 : x and its 1-bit mask
// (bit i = !(y_i <= 0), 8 elements per byte, little-endian; bytes ceil(n/8) ..
// bits_bytes - 1 are zeroed); backward dx_i = bit i ? dy_i : 0.
int launch_relu_fwd(int dtype, const void *x, int64_t n, void *y, void *bits, int64_t bits_bytes, void *stream);
int launch_relu_bwd(int dtype, const void *dy, const void *bits, int64_t n, void *dx, void *stream);

// Dropout over n elements in memory order, forward (in = x) or backward
// (in = dy): out_i = in_i * (u_i >= thresh ? scale : 0), or 0 when drop_all;
// u_i is word i mod 4 of the Philox4x32-10 block with counter
// (b mod 2^32, b div 2^32, 0, 0), b = offset + floor(i / 4), key = seed.
int launch_dropout(int dtype, const void *in, int64_t n, void *out, uint64_t seed, uint64_t offset, uint32_t thresh,
                   float scale, int drop_all, void *stream);

// Global average pool x[N][L][C] -> y[N][C] and its adjoint.
int launch_avgpool_fwd(int dtype, const void *x, int N, int L, int C, void *y, void *stream);
int launch_avgpool_bwd(int dtype, const void *dy, int N, int L, int C, void *dx, void *stream);

// dst[i] = src[i] over a 4-D index space of extents ext, each side with its
// own element strides (layout.hip): the staging of a caller tensor into (or
// out of) the dense layout the kernels read.  dst must not overlap itself
// or src.
int launch_copy4(int dtype, const void *src, const int64_t ext[4], const int64_t sstride[4], void *dst,
                 const int64_t dstride[4], void *stream);

// Per-stream transient workspace (workspace.hip).  Returns null and sets
// *err on failure.
void *workspace_get(void *stream, size_t bytes, int *err);
// Test hook: make the next `n` workspace growths fail.
void workspace_fail_next(int n);

// Fixed scratch of the no-allocation backward (workspace.hip): a static
// device array of kScratchBytes per GPU.  scratch_get returns its device
// address on the current device (looked up once per device) or null with
// *err = 1 when `bytes` exceeds kScratchBytes, 2 on a HIP error.  Every
// caller on one device shares the same bytes.
constexpr size_t kScratchBytes = size_t(64) << 20;
void *scratch_get(size_t bytes, int *err);

int device_last_error();  // hipGetLastError()

// Kernel timing (profile.hip): prof_mark(kind, stream, true) before a launch
// and (.., false) after it record an event pair when `kind` is armed.
enum ProfKind : unsigned {
    kProfFwd = 1u, kProfDgrad = 2u, kProfWgrad = 4u, kProfBn = 8u, kProfAct = 16u, kProfRed = 32u
};
void prof_mark(unsigned kind, void *stream, bool begin);
// For a launch that records its own events (hipExtLaunchKernelGGL stamps the
// dispatch's start and end, so the pair spans the kernel alone, not the
// dispatch latency around it): prof_pair hands out a pair (hipEvent_t) when
// `kind` is armed, and prof_pair_done files it after the launch (or returns
// it to the pool when the launch failed).
bool prof_pair(unsigned kind, void **begin, void **end);
void prof_pair_done(unsigned kind, void *begin, void *end, bool launched);
// Skip prof_mark and prof_pair on the calling thread while `off` (the
// no-allocation backward records no events).
void prof_thread_off(bool off);
int prof_start(unsigned kinds);
int prof_read(unsigned kind, uint64_t *launches, double *total_ms);

}  // namespace ms

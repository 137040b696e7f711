/*
 * CPU oracle for the selective-differentiation layers (TEST INFRASTRUCTURE).
 *
 * This file is the plain, slow, obviously correct definition of what the
 * GPU path computes: the value and the vector-Jacobian products of the three
 * layers that are linear in both their input and their parameters
 * (Sec. 2.2.1: convolution Z = W * X + b, the fully-connected layer
 * y = W x + b of App. C, and batch normalisation in evaluation mode,
 * y = W (x - mu_hat) / sqrt(sigma_hat^2 + eps) + b of App. C), the
 * transposed convolution that Sec. 2.2.1 and App. B name beside them (in 2-D
 * and 3-D), the
 * dropout of Sec. 2.2.2 with its counter-based generator, plus the
 * parameter-free global average pool used to shape the ResNet-18-like stack.
 *
 * Only tests/, __graft_entry__.smoke() and the cpu_baseline leg of bench.py
 * may load or call this code.  It shares nothing with the HIP library: no
 * header, helper, table or constant.  Every array is a dense row-major
 * float64 array in the logical PyTorch order (conv/BN: N,C,H,W; conv weight:
 * K,C,R,S; linear: X[M,K_in], W[N_out,K_in]).  Every sum is accumulated in
 * float64 in the ascending order of its indices; outputs stay float64 and
 * orc_round() rounds them once to a storage precision when a caller needs it.
 *
 * Convolution is cross-correlation with zero padding, dilation 1, groups 1,
 * as torch.nn.Conv2d computes it (the '*' of Sec. 2.2.1 is read that way).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

typedef int64_t i64;

#define IDX4(a, b, c, d, B, C, D) ((((a) * (B) + (b)) * (C) + (c)) * (D) + (d))

static i64 out_extent(i64 in, i64 pad, i64 k, i64 stride)
{
    return (in + 2 * pad - k) / stride + 1;
}

/* ---------------------------------------------------------------------------
 * Conv2d forward (Sec. 2.2.1, Z = W * X + b):
 *   y[n,k,p,q] = b[k] + sum_{c,r,s} W[k,c,r,s] * x[n,c, p*sh-ph+r, q*sw-pw+s]
 * with x taken as zero outside [0,H) x [0,W).  b may be NULL (no bias).
 * ------------------------------------------------------------------------- */
static double conv_fwd_one(const double *x, const double *w, const double *b,
                           i64 n, i64 k, i64 p, i64 q,
                           i64 C, i64 H, i64 W, i64 R, i64 S,
                           i64 sh, i64 sw, i64 ph, i64 pw)
{
    double acc = 0.0;
    for (i64 c = 0; c < C; ++c)
        for (i64 r = 0; r < R; ++r) {
            i64 ih = p * sh - ph + r;
            if (ih < 0 || ih >= H) continue;
            for (i64 s = 0; s < S; ++s) {
                i64 iw = q * sw - pw + s;
                if (iw < 0 || iw >= W) continue;
                acc += w[IDX4(k, c, r, s, C, R, S)] * x[IDX4(n, c, ih, iw, C, H, W)];
            }
        }
    return acc + (b ? b[k] : 0.0);
}

void orc_conv2d_forward(const double *x, const double *w, const double *b, double *y,
                        i64 N, i64 C, i64 H, i64 W, i64 K, i64 R, i64 S,
                        i64 sh, i64 sw, i64 ph, i64 pw)
{
    i64 P = out_extent(H, ph, R, sh), Q = out_extent(W, pw, S, sw);
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 n = 0; n < N; ++n)
        for (i64 k = 0; k < K; ++k)
            for (i64 p = 0; p < P; ++p)
                for (i64 q = 0; q < Q; ++q)
                    y[IDX4(n, k, p, q, K, P, Q)] =
                        conv_fwd_one(x, w, b, n, k, p, q, C, H, W, R, S, sh, sw, ph, pw);
}

/* The same value at `count` sampled output coordinates idx[4*i..4*i+3] =
 * (n, k, p, q). */
void orc_conv2d_forward_at(const double *x, const double *w, const double *b,
                           i64 N, i64 C, i64 H, i64 W, i64 K, i64 R, i64 S,
                           i64 sh, i64 sw, i64 ph, i64 pw,
                           const i64 *idx, i64 count, double *out)
{
    (void)N; (void)K;
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < count; ++i)
        out[i] = conv_fwd_one(x, w, b, idx[4 * i], idx[4 * i + 1], idx[4 * i + 2],
                              idx[4 * i + 3], C, H, W, R, S, sh, sw, ph, pw);
}

/* ---------------------------------------------------------------------------
 * Conv2d input gradient (Sec. 2.2.1: the input Jacobian depends on W only).
 * Written as the adjoint of the forward map: every product the forward adds
 * into y[n,k,p,q] from x[n,c,ih,iw] sends W[k,c,r,s] * dy[n,k,p,q] back to
 * dx[n,c,ih,iw].
 * ------------------------------------------------------------------------- */
void orc_conv2d_input_grad(const double *dy, const double *w, double *dx,
                           i64 N, i64 C, i64 H, i64 W, i64 K, i64 R, i64 S,
                           i64 sh, i64 sw, i64 ph, i64 pw)
{
    i64 P = out_extent(H, ph, R, sh), Q = out_extent(W, pw, S, sw);
#pragma omp parallel for schedule(static)
    for (i64 n = 0; n < N; ++n) {
        double *dxn = dx + n * C * H * W;
        memset(dxn, 0, sizeof(double) * (size_t)(C * H * W));
        for (i64 k = 0; k < K; ++k)
            for (i64 p = 0; p < P; ++p)
                for (i64 q = 0; q < Q; ++q) {
                    double g = dy[IDX4(n, k, p, q, K, P, Q)];
                    for (i64 c = 0; c < C; ++c)
                        for (i64 r = 0; r < R; ++r) {
                            i64 ih = p * sh - ph + r;
                            if (ih < 0 || ih >= H) continue;
                            for (i64 s = 0; s < S; ++s) {
                                i64 iw = q * sw - pw + s;
                                if (iw < 0 || iw >= W) continue;
                                dxn[(c * H + ih) * W + iw] += w[IDX4(k, c, r, s, C, R, S)] * g;
                            }
                        }
                }
    }
}

/* One input-gradient entry dx[n,c,h,w], gathered: the sum over (k,r,s) of
 * W[k,c,r,s] * dy[n,k,p,q] for the output positions (p,q) whose receptive
 * field covers (h,w) through tap (r,s), i.e. p*sh - ph + r = h. */
void orc_conv2d_input_grad_at(const double *dy, const double *w,
                              i64 N, i64 C, i64 H, i64 W, i64 K, i64 R, i64 S,
                              i64 sh, i64 sw, i64 ph, i64 pw,
                              const i64 *idx, i64 count, double *out)
{
    (void)N;
    i64 P = out_extent(H, ph, R, sh), Q = out_extent(W, pw, S, sw);
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < count; ++i) {
        i64 n = idx[4 * i], c = idx[4 * i + 1], h = idx[4 * i + 2], x = idx[4 * i + 3];
        double acc = 0.0;
        for (i64 k = 0; k < K; ++k)
            for (i64 r = 0; r < R; ++r) {
                i64 th = h + ph - r;
                if (th < 0 || th % sh != 0) continue;
                i64 p = th / sh;
                if (p >= P) continue;
                for (i64 s = 0; s < S; ++s) {
                    i64 tw = x + pw - s;
                    if (tw < 0 || tw % sw != 0) continue;
                    i64 q = tw / sw;
                    if (q >= Q) continue;
                    acc += w[IDX4(k, c, r, s, C, R, S)] * dy[IDX4(n, k, p, q, K, P, Q)];
                }
            }
        out[i] = acc;
    }
}

/* ---------------------------------------------------------------------------
 * Conv2d weight gradient (Sec. 2.2.1: the weight Jacobian depends on X only):
 *   dW[k,c,r,s] = sum_{n,p,q} dy[n,k,p,q] * x[n,c, p*sh-ph+r, q*sw-pw+s]
 * ------------------------------------------------------------------------- */
static double conv_wgrad_one(const double *dy, const double *x,
                             i64 k, i64 c, i64 r, i64 s,
                             i64 N, i64 C, i64 H, i64 W, i64 K, i64 P, i64 Q,
                             i64 sh, i64 sw, i64 ph, i64 pw)
{
    double acc = 0.0;
    for (i64 n = 0; n < N; ++n)
        for (i64 p = 0; p < P; ++p) {
            i64 ih = p * sh - ph + r;
            if (ih < 0 || ih >= H) continue;
            for (i64 q = 0; q < Q; ++q) {
                i64 iw = q * sw - pw + s;
                if (iw < 0 || iw >= W) continue;
                acc += dy[IDX4(n, k, p, q, K, P, Q)] * x[IDX4(n, c, ih, iw, C, H, W)];
            }
        }
    return acc;
}

void orc_conv2d_weight_grad(const double *dy, const double *x, double *dw,
                            i64 N, i64 C, i64 H, i64 W, i64 K, i64 R, i64 S,
                            i64 sh, i64 sw, i64 ph, i64 pw)
{
    i64 P = out_extent(H, ph, R, sh), Q = out_extent(W, pw, S, sw);
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 k = 0; k < K; ++k)
        for (i64 c = 0; c < C; ++c)
            for (i64 r = 0; r < R; ++r)
                for (i64 s = 0; s < S; ++s)
                    dw[IDX4(k, c, r, s, C, R, S)] =
                        conv_wgrad_one(dy, x, k, c, r, s, N, C, H, W, K, P, Q, sh, sw, ph, pw);
}

/* Sampled weight-gradient entries, idx[4*i..] = (k, c, r, s). */
void orc_conv2d_weight_grad_at(const double *dy, const double *x,
                               i64 N, i64 C, i64 H, i64 W, i64 K, i64 R, i64 S,
                               i64 sh, i64 sw, i64 ph, i64 pw,
                               const i64 *idx, i64 count, double *out)
{
    i64 P = out_extent(H, ph, R, sh), Q = out_extent(W, pw, S, sw);
#pragma omp parallel for schedule(dynamic, 16)
    for (i64 i = 0; i < count; ++i)
        out[i] = conv_wgrad_one(dy, x, idx[4 * i], idx[4 * i + 1], idx[4 * i + 2],
                                idx[4 * i + 3], N, C, H, W, K, P, Q, sh, sw, ph, pw);
}

/* Conv2d bias gradient (Sec. 2.2.1: no dependency): db[k] = sum_{n,p,q} dy. */
void orc_conv2d_bias_grad(const double *dy, double *db, i64 N, i64 K, i64 P, i64 Q)
{
#pragma omp parallel for schedule(static)
    for (i64 k = 0; k < K; ++k) {
        double acc = 0.0;
        for (i64 n = 0; n < N; ++n)
            for (i64 p = 0; p < P; ++p)
                for (i64 q = 0; q < Q; ++q)
                    acc += dy[IDX4(n, k, p, q, K, P, Q)];
        db[k] = acc;
    }
}

/* ---------------------------------------------------------------------------
 * Transposed convolution (the (transpose) convolution of Sec. 2.2.1 and the
 * ConvTransposeNd of App. B), as torch.nn.ConvTranspose2d defines it with
 * dilation 1 and groups 1: x[N,Ci,H,W], W[Ci,Co,R,S], output
 * [N,Co,Ho,Wo] with Ho = (H-1) sh - 2 ph + R + oph (likewise Wo).  Every
 * input pixel (h,w) scatters x[n,i,h,w] W[i,o,r,s] to the output pixel
 * (h sh - ph + r, w sw - pw + s) when that lies inside the output:
 *   y[n,o,h',w'] = b[o] + sum over (i,h,w,r,s) with h sh - ph + r = h' and
 *                  w sw - pw + s = w' of x[n,i,h,w] W[i,o,r,s].
 * The layer is linear in x and in W, so the rule of Sec. 2.2.1 applies: the
 * input gradient needs W only, the weight gradient x only.
 * ------------------------------------------------------------------------- */
void orc_convt2d_forward(const double *x, const double *w, const double *b, double *y,
                         i64 N, i64 Ci, i64 H, i64 W, i64 Co, i64 R, i64 S,
                         i64 sh, i64 sw, i64 ph, i64 pw, i64 Ho, i64 Wo)
{
#pragma omp parallel for schedule(static)
    for (i64 n = 0; n < N; ++n) {
        double *yn = y + n * Co * Ho * Wo;
        for (i64 o = 0; o < Co; ++o)
            for (i64 t = 0; t < Ho * Wo; ++t)
                yn[o * Ho * Wo + t] = b ? b[o] : 0.0;
        for (i64 i = 0; i < Ci; ++i)
            for (i64 h = 0; h < H; ++h)
                for (i64 ww = 0; ww < W; ++ww) {
                    double xv = x[IDX4(n, i, h, ww, Ci, H, W)];
                    for (i64 o = 0; o < Co; ++o)
                        for (i64 r = 0; r < R; ++r) {
                            i64 oh = h * sh - ph + r;
                            if (oh < 0 || oh >= Ho) continue;
                            for (i64 s = 0; s < S; ++s) {
                                i64 ow = ww * sw - pw + s;
                                if (ow < 0 || ow >= Wo) continue;
                                yn[(o * Ho + oh) * Wo + ow] += xv * w[IDX4(i, o, r, s, Co, R, S)];
                            }
                        }
                }
    }
}

/* One output entry y[n,o,h',w'], gathered: the taps (r,s) and input pixels
 * (h,w) with h sh - ph + r = h' (h an integer in [0,H)), likewise for w. */
void orc_convt2d_forward_at(const double *x, const double *w, const double *b,
                            i64 N, i64 Ci, i64 H, i64 W, i64 Co, i64 R, i64 S,
                            i64 sh, i64 sw, i64 ph, i64 pw,
                            const i64 *idx, i64 count, double *out)
{
    (void)N;
#pragma omp parallel for schedule(static)
    for (i64 k = 0; k < count; ++k) {
        i64 n = idx[4 * k], o = idx[4 * k + 1], oh = idx[4 * k + 2], ow = idx[4 * k + 3];
        double acc = 0.0;
        for (i64 i = 0; i < Ci; ++i)
            for (i64 r = 0; r < R; ++r) {
                i64 th = oh + ph - r;
                if (th < 0 || th % sh != 0 || th / sh >= H) continue;
                for (i64 s = 0; s < S; ++s) {
                    i64 tw = ow + pw - s;
                    if (tw < 0 || tw % sw != 0 || tw / sw >= W) continue;
                    acc += x[IDX4(n, i, th / sh, tw / sw, Ci, H, W)] * w[IDX4(i, o, r, s, Co, R, S)];
                }
            }
        out[k] = acc + (b ? b[o] : 0.0);
    }
}

/* Input gradient: each scattered product x[n,i,h,w] W[i,o,r,s] sends
 * W[i,o,r,s] dy[n,o,h',w'] back to x[n,i,h,w], so
 *   dx[n,i,h,w] = sum_{o,r,s} W[i,o,r,s] dy[n,o, h sh - ph + r, w sw - pw + s]
 * over the output pixels inside [0,Ho) x [0,Wo). */
static double convt_dgrad_one(const double *dy, const double *w, i64 n, i64 i, i64 h, i64 ww,
                              i64 Co, i64 R, i64 S, i64 sh, i64 sw, i64 ph, i64 pw, i64 Ho, i64 Wo)
{
    double acc = 0.0;
    for (i64 o = 0; o < Co; ++o)
        for (i64 r = 0; r < R; ++r) {
            i64 oh = h * sh - ph + r;
            if (oh < 0 || oh >= Ho) continue;
            for (i64 s = 0; s < S; ++s) {
                i64 ow = ww * sw - pw + s;
                if (ow < 0 || ow >= Wo) continue;
                acc += w[IDX4(i, o, r, s, Co, R, S)] * dy[IDX4(n, o, oh, ow, Co, Ho, Wo)];
            }
        }
    return acc;
}

void orc_convt2d_input_grad(const double *dy, const double *w, double *dx,
                            i64 N, i64 Ci, i64 H, i64 W, i64 Co, i64 R, i64 S,
                            i64 sh, i64 sw, i64 ph, i64 pw, i64 Ho, i64 Wo)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 n = 0; n < N; ++n)
        for (i64 i = 0; i < Ci; ++i)
            for (i64 h = 0; h < H; ++h)
                for (i64 ww = 0; ww < W; ++ww)
                    dx[IDX4(n, i, h, ww, Ci, H, W)] =
                        convt_dgrad_one(dy, w, n, i, h, ww, Co, R, S, sh, sw, ph, pw, Ho, Wo);
}

void orc_convt2d_input_grad_at(const double *dy, const double *w,
                               i64 N, i64 Ci, i64 H, i64 W, i64 Co, i64 R, i64 S,
                               i64 sh, i64 sw, i64 ph, i64 pw, i64 Ho, i64 Wo,
                               const i64 *idx, i64 count, double *out)
{
    (void)N; (void)Ci; (void)H; (void)W;
#pragma omp parallel for schedule(static)
    for (i64 k = 0; k < count; ++k)
        out[k] = convt_dgrad_one(dy, w, idx[4 * k], idx[4 * k + 1], idx[4 * k + 2], idx[4 * k + 3],
                                 Co, R, S, sh, sw, ph, pw, Ho, Wo);
}

/* Weight gradient:
 *   dW[i,o,r,s] = sum_{n,h,w} x[n,i,h,w] dy[n,o, h sh - ph + r, w sw - pw + s]
 * over the output pixels inside [0,Ho) x [0,Wo). */
static double convt_wgrad_one(const double *dy, const double *x, i64 i, i64 o, i64 r, i64 s,
                              i64 N, i64 Ci, i64 H, i64 W, i64 Co,
                              i64 sh, i64 sw, i64 ph, i64 pw, i64 Ho, i64 Wo)
{
    double acc = 0.0;
    for (i64 n = 0; n < N; ++n)
        for (i64 h = 0; h < H; ++h) {
            i64 oh = h * sh - ph + r;
            if (oh < 0 || oh >= Ho) continue;
            for (i64 ww = 0; ww < W; ++ww) {
                i64 ow = ww * sw - pw + s;
                if (ow < 0 || ow >= Wo) continue;
                acc += x[IDX4(n, i, h, ww, Ci, H, W)] * dy[IDX4(n, o, oh, ow, Co, Ho, Wo)];
            }
        }
    return acc;
}

void orc_convt2d_weight_grad(const double *dy, const double *x, double *dw,
                             i64 N, i64 Ci, i64 H, i64 W, i64 Co, i64 R, i64 S,
                             i64 sh, i64 sw, i64 ph, i64 pw, i64 Ho, i64 Wo)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 i = 0; i < Ci; ++i)
        for (i64 o = 0; o < Co; ++o)
            for (i64 r = 0; r < R; ++r)
                for (i64 s = 0; s < S; ++s)
                    dw[IDX4(i, o, r, s, Co, R, S)] =
                        convt_wgrad_one(dy, x, i, o, r, s, N, Ci, H, W, Co, sh, sw, ph, pw, Ho, Wo);
}

void orc_convt2d_weight_grad_at(const double *dy, const double *x,
                                i64 N, i64 Ci, i64 H, i64 W, i64 Co, i64 R, i64 S,
                                i64 sh, i64 sw, i64 ph, i64 pw, i64 Ho, i64 Wo,
                                const i64 *idx, i64 count, double *out)
{
    (void)R; (void)S;
#pragma omp parallel for schedule(dynamic, 16)
    for (i64 k = 0; k < count; ++k)
        out[k] = convt_wgrad_one(dy, x, idx[4 * k], idx[4 * k + 1], idx[4 * k + 2], idx[4 * k + 3],
                                 N, Ci, H, W, Co, sh, sw, ph, pw, Ho, Wo);
}

/* ---------------------------------------------------------------------------
 * 3-D convolution and its transpose (App. B probes torch.nn.Conv3d and
 * torch.nn.ConvTranspose3d): the 2-D definitions with a depth axis added.
 * Arrays are dense in logical order: x[N,C,D,H,W], conv weight W[K,C,T,R,S],
 * transposed weight W[Ci,Co,T,R,S].  g3 packs the geometry:
 *   g3 = {N, C, D, H, W, K, T, R, S, Do, P, Q, sd, sh, sw, pd, ph, pw}
 * where (Do, P, Q) is the convolution's output extent (the transposed
 * layer's input extent is (D, H, W) of its adjoint convolution's output).
 * ------------------------------------------------------------------------- */
#define IDX5(a, b, c, d, e, B, C, D, E) (((((a) * (B) + (b)) * (C) + (c)) * (D) + (d)) * (E) + (e))

/* y[n,k,o,p,q] = b[k] + sum_{c,t,r,s} W[k,c,t,r,s] x[n,c,o sd-pd+t, p sh-ph+r, q sw-pw+s] */
static double conv3d_fwd_one(const double *x, const double *w, const double *b, const i64 *g,
                             i64 n, i64 k, i64 o, i64 p, i64 q)
{
    i64 C = g[1], D = g[2], H = g[3], W = g[4], T = g[6], R = g[7], S = g[8];
    double acc = 0.0;
    for (i64 c = 0; c < C; ++c)
        for (i64 t = 0; t < T; ++t) {
            i64 id = o * g[12] - g[15] + t;
            if (id < 0 || id >= D) continue;
            for (i64 r = 0; r < R; ++r) {
                i64 ih = p * g[13] - g[16] + r;
                if (ih < 0 || ih >= H) continue;
                for (i64 s = 0; s < S; ++s) {
                    i64 iw = q * g[14] - g[17] + s;
                    if (iw < 0 || iw >= W) continue;
                    acc += w[IDX5(k, c, t, r, s, C, T, R, S)] * x[IDX5(n, c, id, ih, iw, C, D, H, W)];
                }
            }
        }
    return acc + (b ? b[k] : 0.0);
}

void orc_conv3d_forward(const double *x, const double *w, const double *b, double *y, const i64 *g)
{
    i64 N = g[0], K = g[5], Do = g[9], P = g[10], Q = g[11];
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 n = 0; n < N; ++n)
        for (i64 k = 0; k < K; ++k)
            for (i64 o = 0; o < Do; ++o)
                for (i64 p = 0; p < P; ++p)
                    for (i64 q = 0; q < Q; ++q)
                        y[IDX5(n, k, o, p, q, K, Do, P, Q)] = conv3d_fwd_one(x, w, b, g, n, k, o, p, q);
}

/* dx[n,c,d,h,w] = sum over (k,t,r,s) and output positions (o,p,q) with
 * o sd-pd+t = d, p sh-ph+r = h, q sw-pw+s = w of W[k,c,t,r,s] dy[n,k,o,p,q] */
void orc_conv3d_input_grad(const double *dy, const double *w, double *dx, const i64 *g)
{
    i64 N = g[0], C = g[1], D = g[2], H = g[3], W = g[4], K = g[5], T = g[6], R = g[7], S = g[8];
    i64 Do = g[9], P = g[10], Q = g[11];
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 n = 0; n < N; ++n)
        for (i64 c = 0; c < C; ++c)
            for (i64 d = 0; d < D; ++d)
                for (i64 h = 0; h < H; ++h)
                    for (i64 ww = 0; ww < W; ++ww) {
                        double acc = 0.0;
                        for (i64 k = 0; k < K; ++k)
                            for (i64 t = 0; t < T; ++t) {
                                i64 td = d + g[15] - t;
                                if (td < 0 || td % g[12] != 0 || td / g[12] >= Do) continue;
                                for (i64 r = 0; r < R; ++r) {
                                    i64 th = h + g[16] - r;
                                    if (th < 0 || th % g[13] != 0 || th / g[13] >= P) continue;
                                    for (i64 s = 0; s < S; ++s) {
                                        i64 tw = ww + g[17] - s;
                                        if (tw < 0 || tw % g[14] != 0 || tw / g[14] >= Q) continue;
                                        acc += w[IDX5(k, c, t, r, s, C, T, R, S)] *
                                               dy[IDX5(n, k, td / g[12], th / g[13], tw / g[14], K, Do, P, Q)];
                                    }
                                }
                            }
                        dx[IDX5(n, c, d, h, ww, C, D, H, W)] = acc;
                    }
}

/* dW[k,c,t,r,s] = sum_{n,o,p,q} dy[n,k,o,p,q] x[n,c,o sd-pd+t, p sh-ph+r, q sw-pw+s] */
void orc_conv3d_weight_grad(const double *dy, const double *x, double *dw, const i64 *g)
{
    i64 N = g[0], C = g[1], D = g[2], H = g[3], W = g[4], K = g[5], T = g[6], R = g[7], S = g[8];
    i64 Do = g[9], P = g[10], Q = g[11];
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 k = 0; k < K; ++k)
        for (i64 c = 0; c < C; ++c)
            for (i64 t = 0; t < T; ++t)
                for (i64 r = 0; r < R; ++r)
                    for (i64 s = 0; s < S; ++s) {
                        double acc = 0.0;
                        for (i64 n = 0; n < N; ++n)
                            for (i64 o = 0; o < Do; ++o) {
                                i64 id = o * g[12] - g[15] + t;
                                if (id < 0 || id >= D) continue;
                                for (i64 p = 0; p < P; ++p) {
                                    i64 ih = p * g[13] - g[16] + r;
                                    if (ih < 0 || ih >= H) continue;
                                    for (i64 q = 0; q < Q; ++q) {
                                        i64 iw = q * g[14] - g[17] + s;
                                        if (iw < 0 || iw >= W) continue;
                                        acc += dy[IDX5(n, k, o, p, q, K, Do, P, Q)] * x[IDX5(n, c, id, ih, iw, C, D, H, W)];
                                    }
                                }
                            }
                        dw[IDX5(k, c, t, r, s, C, T, R, S)] = acc;
                    }
}

/* Transposed 3-D convolution, x[N,Ci,D,H,W], W[Ci,Co,T,R,S], output
 * [N,Co,Do,Ho,Wo]: every input voxel scatters x W through each tap to the
 * output voxel (d sd-pd+t, h sh-ph+r, w sw-pw+s) when that lies inside.
 * Here g3 = {N, Ci, D, H, W, Co, T, R, S, Do, Ho, Wo, sd, sh, sw, pd, ph, pw}. */
void orc_convt3d_forward(const double *x, const double *w, const double *b, double *y, const i64 *g)
{
    i64 N = g[0], Ci = g[1], D = g[2], H = g[3], W = g[4], Co = g[5], T = g[6], R = g[7], S = g[8];
    i64 Do = g[9], Ho = g[10], Wo = g[11];
#pragma omp parallel for schedule(static)
    for (i64 n = 0; n < N; ++n) {
        double *yn = y + n * Co * Do * Ho * Wo;
        for (i64 o = 0; o < Co; ++o)
            for (i64 v = 0; v < Do * Ho * Wo; ++v)
                yn[o * Do * Ho * Wo + v] = b ? b[o] : 0.0;
        for (i64 i = 0; i < Ci; ++i)
            for (i64 d = 0; d < D; ++d)
                for (i64 h = 0; h < H; ++h)
                    for (i64 ww = 0; ww < W; ++ww) {
                        double xv = x[IDX5(n, i, d, h, ww, Ci, D, H, W)];
                        for (i64 o = 0; o < Co; ++o)
                            for (i64 t = 0; t < T; ++t) {
                                i64 od = d * g[12] - g[15] + t;
                                if (od < 0 || od >= Do) continue;
                                for (i64 r = 0; r < R; ++r) {
                                    i64 oh = h * g[13] - g[16] + r;
                                    if (oh < 0 || oh >= Ho) continue;
                                    for (i64 s = 0; s < S; ++s) {
                                        i64 ow = ww * g[14] - g[17] + s;
                                        if (ow < 0 || ow >= Wo) continue;
                                        yn[((o * Do + od) * Ho + oh) * Wo + ow] += xv * w[IDX5(i, o, t, r, s, Co, T, R, S)];
                                    }
                                }
                            }
                    }
    }
}

/* dx[n,i,d,h,w] = sum_{o,t,r,s} W[i,o,t,r,s] dy[n,o, d sd-pd+t, h sh-ph+r, w sw-pw+s] */
void orc_convt3d_input_grad(const double *dy, const double *w, double *dx, const i64 *g)
{
    i64 N = g[0], Ci = g[1], D = g[2], H = g[3], W = g[4], Co = g[5], T = g[6], R = g[7], S = g[8];
    i64 Do = g[9], Ho = g[10], Wo = g[11];
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 n = 0; n < N; ++n)
        for (i64 i = 0; i < Ci; ++i)
            for (i64 d = 0; d < D; ++d)
                for (i64 h = 0; h < H; ++h)
                    for (i64 ww = 0; ww < W; ++ww) {
                        double acc = 0.0;
                        for (i64 o = 0; o < Co; ++o)
                            for (i64 t = 0; t < T; ++t) {
                                i64 od = d * g[12] - g[15] + t;
                                if (od < 0 || od >= Do) continue;
                                for (i64 r = 0; r < R; ++r) {
                                    i64 oh = h * g[13] - g[16] + r;
                                    if (oh < 0 || oh >= Ho) continue;
                                    for (i64 s = 0; s < S; ++s) {
                                        i64 ow = ww * g[14] - g[17] + s;
                                        if (ow < 0 || ow >= Wo) continue;
                                        acc += w[IDX5(i, o, t, r, s, Co, T, R, S)] * dy[IDX5(n, o, od, oh, ow, Co, Do, Ho, Wo)];
                                    }
                                }
                            }
                        dx[IDX5(n, i, d, h, ww, Ci, D, H, W)] = acc;
                    }
}

/* dW[i,o,t,r,s] = sum_{n,d,h,w} x[n,i,d,h,w] dy[n,o, d sd-pd+t, h sh-ph+r, w sw-pw+s] */
void orc_convt3d_weight_grad(const double *dy, const double *x, double *dw, const i64 *g)
{
    i64 N = g[0], Ci = g[1], D = g[2], H = g[3], W = g[4], Co = g[5], T = g[6], R = g[7], S = g[8];
    i64 Do = g[9], Ho = g[10], Wo = g[11];
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 i = 0; i < Ci; ++i)
        for (i64 o = 0; o < Co; ++o)
            for (i64 t = 0; t < T; ++t)
                for (i64 r = 0; r < R; ++r)
                    for (i64 s = 0; s < S; ++s) {
                        double acc = 0.0;
                        for (i64 n = 0; n < N; ++n)
                            for (i64 d = 0; d < D; ++d) {
                                i64 od = d * g[12] - g[15] + t;
                                if (od < 0 || od >= Do) continue;
                                for (i64 h = 0; h < H; ++h) {
                                    i64 oh = h * g[13] - g[16] + r;
                                    if (oh < 0 || oh >= Ho) continue;
                                    for (i64 ww = 0; ww < W; ++ww) {
                                        i64 ow = ww * g[14] - g[17] + s;
                                        if (ow < 0 || ow >= Wo) continue;
                                        acc += x[IDX5(n, i, d, h, ww, Ci, D, H, W)] * dy[IDX5(n, o, od, oh, ow, Co, Do, Ho, Wo)];
                                    }
                                }
                            }
                        dw[IDX5(i, o, t, r, s, Co, T, R, S)] = acc;
                    }
}

/* Bias gradient of a 5-D output: db[k] = sum over (n, o, p, q) of dy. */
void orc_bias_grad5(const double *dy, double *db, i64 N, i64 K, i64 V)
{
#pragma omp parallel for schedule(static)
    for (i64 k = 0; k < K; ++k) {
        double acc = 0.0;
        for (i64 n = 0; n < N; ++n)
            for (i64 v = 0; v < V; ++v) acc += dy[(n * K + k) * V + v];
        db[k] = acc;
    }
}

/* ---------------------------------------------------------------------------
 * Dropout that regenerates its mask (Sec. 2.2.2): instead of the mask, the
 * layer keeps the state of a counter-based generator and draws the mask
 * again in backward.  The generator is Philox4x32 with 10 rounds (Salmon,
 * Moraes, Dror and Shaw, "Parallel random numbers: as easy as 1, 2, 3",
 * SC 2011): a 128-bit counter c0..c3 and a 64-bit key k0, k1; each round
 * multiplies c0 and c2 by two fixed 32-bit constants, mixes the high halves
 * of the products with the other two words and the key, and the key is
 * bumped by two Weyl constants between rounds.
 *
 * The stream of a call: element i (memory order) takes word i mod 4 of the
 * block with counter (b mod 2^32, b div 2^32, 0, 0), b = offset + floor(i/4),
 * key (seed mod 2^32, seed div 2^32).  It is kept iff that word is >= thresh.
 * ------------------------------------------------------------------------- */
static uint32_t mulhi32(uint32_t a, uint32_t b, uint32_t *lo)
{
    uint64_t p = (uint64_t)a * (uint64_t)b;
    *lo = (uint32_t)p;
    return (uint32_t)(p >> 32);
}

void orc_philox4x32_10(const uint32_t *ctr, const uint32_t *key, uint32_t *out)
{
    const uint32_t mul0 = 0xD2511F53u, mul1 = 0xCD9E8D57u;      /* round multipliers */
    const uint32_t weyl0 = 0x9E3779B9u, weyl1 = 0xBB67AE85u;    /* key increments    */
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        uint32_t lo0, lo1;
        uint32_t hi0 = mulhi32(mul0, c0, &lo0);
        uint32_t hi1 = mulhi32(mul1, c2, &lo1);
        uint32_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += weyl0;
        k1 += weyl1;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The stream words u_i of a call, i < n. */
void orc_dropout_words(i64 n, uint64_t seed, uint64_t offset, uint32_t *u)
{
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
#pragma omp parallel for schedule(static)
    for (i64 blk = 0; blk < (n + 3) / 4; ++blk) {
        uint64_t b = offset + (uint64_t)blk;
        const uint32_t ctr[4] = {(uint32_t)b, (uint32_t)(b >> 32), 0u, 0u};
        uint32_t w[4];
        orc_philox4x32_10(ctr, key, w);
        for (int j = 0; j < 4 && 4 * blk + j < n; ++j) u[4 * blk + j] = w[j];
    }
}

/* ---------------------------------------------------------------------------
 * Fully-connected layer (App. C, y = W x + b, applied to every row of X):
 *   Y[m,j]  = b[j] + sum_i X[m,i] W[j,i]
 *   dX[m,i] = sum_j dY[m,j] W[j,i]          (needs W only)
 *   dW[j,i] = sum_m dY[m,j] X[m,i]          (needs X only)
 *   db[j]   = sum_m dY[m,j]                 (needs nothing)
 * ------------------------------------------------------------------------- */
static double lin_fwd_one(const double *X, const double *Wt, const double *b,
                          i64 m, i64 j, i64 Kin)
{
    double acc = 0.0;
    for (i64 i = 0; i < Kin; ++i) acc += X[m * Kin + i] * Wt[j * Kin + i];
    return acc + (b ? b[j] : 0.0);
}

void orc_linear_forward(const double *X, const double *Wt, const double *b, double *Y,
                        i64 M, i64 Kin, i64 Nout)
{
#pragma omp parallel for schedule(static)
    for (i64 m = 0; m < M; ++m)
        for (i64 j = 0; j < Nout; ++j) Y[m * Nout + j] = lin_fwd_one(X, Wt, b, m, j, Kin);
}

void orc_linear_forward_at(const double *X, const double *Wt, const double *b,
                           i64 M, i64 Kin, i64 Nout, const i64 *idx, i64 count, double *out)
{
    (void)M; (void)Nout;
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < count; ++i) out[i] = lin_fwd_one(X, Wt, b, idx[2 * i], idx[2 * i + 1], Kin);
}

static double lin_dgrad_one(const double *dY, const double *Wt, i64 m, i64 i, i64 Kin, i64 Nout)
{
    double acc = 0.0;
    for (i64 j = 0; j < Nout; ++j) acc += dY[m * Nout + j] * Wt[j * Kin + i];
    return acc;
}

void orc_linear_input_grad(const double *dY, const double *Wt, double *dX,
                           i64 M, i64 Kin, i64 Nout)
{
#pragma omp parallel for schedule(static)
    for (i64 m = 0; m < M; ++m)
        for (i64 i = 0; i < Kin; ++i) dX[m * Kin + i] = lin_dgrad_one(dY, Wt, m, i, Kin, Nout);
}

void orc_linear_input_grad_at(const double *dY, const double *Wt, i64 M, i64 Kin, i64 Nout,
                              const i64 *idx, i64 count, double *out)
{
    (void)M;
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < count; ++i) out[i] = lin_dgrad_one(dY, Wt, idx[2 * i], idx[2 * i + 1], Kin, Nout);
}

static double lin_wgrad_one(const double *dY, const double *X, i64 j, i64 i,
                            i64 M, i64 Kin, i64 Nout)
{
    double acc = 0.0;
    for (i64 m = 0; m < M; ++m) acc += dY[m * Nout + j] * X[m * Kin + i];
    return acc;
}

void orc_linear_weight_grad(const double *dY, const double *X, double *dW,
                            i64 M, i64 Kin, i64 Nout)
{
#pragma omp parallel for schedule(static)
    for (i64 j = 0; j < Nout; ++j)
        for (i64 i = 0; i < Kin; ++i) dW[j * Kin + i] = lin_wgrad_one(dY, X, j, i, M, Kin, Nout);
}

void orc_linear_weight_grad_at(const double *dY, const double *X, i64 M, i64 Kin, i64 Nout,
                               const i64 *idx, i64 count, double *out)
{
#pragma omp parallel for schedule(dynamic, 16)
    for (i64 i = 0; i < count; ++i)
        out[i] = lin_wgrad_one(dY, X, idx[2 * i], idx[2 * i + 1], M, Kin, Nout);
}

void orc_linear_bias_grad(const double *dY, double *db, i64 M, i64 Nout)
{
#pragma omp parallel for schedule(static)
    for (i64 j = 0; j < Nout; ++j) {
        double acc = 0.0;
        for (i64 m = 0; m < M; ++m) acc += dY[m * Nout + j];
        db[j] = acc;
    }
}

/* ---------------------------------------------------------------------------
 * Batch normalisation in evaluation mode (App. C):
 *   y = gamma * (x - mu_hat) / sqrt(sigma_hat^2 + eps) + beta
 * per channel c of x[N, C, L] (L = H*W; L = 1 for a [N, C] input), with the
 * running statistics mu_hat, sigma_hat^2 fixed buffers.  gamma == NULL means
 * gamma = 1 and beta == NULL means beta = 0 (affine=False).
 * Backward (the map is affine in x, gamma and beta):
 *   dx     = dy * gamma / sqrt(sigma_hat^2 + eps)              (no x needed)
 *   dgamma = sum_{n,l} dy * (x - mu_hat) / sqrt(sigma_hat^2 + eps)
 *   dbeta  = sum_{n,l} dy
 * Any of dx, dgamma, dbeta may be NULL to skip it.
 * ------------------------------------------------------------------------- */
void orc_bn_eval_forward(const double *x, const double *mean, const double *var,
                         const double *gamma, const double *beta, double eps, double *y,
                         i64 N, i64 C, i64 L)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 n = 0; n < N; ++n)
        for (i64 c = 0; c < C; ++c) {
            double g = gamma ? gamma[c] : 1.0, bt = beta ? beta[c] : 0.0;
            for (i64 l = 0; l < L; ++l) {
                i64 o = (n * C + c) * L + l;
                y[o] = g * (x[o] - mean[c]) / sqrt(var[c] + eps) + bt;
            }
        }
}

void orc_bn_eval_backward(const double *dy, const double *x, const double *mean,
                          const double *var, const double *gamma, double eps,
                          double *dx, double *dgamma, double *dbeta,
                          i64 N, i64 C, i64 L)
{
    if (dx) {
#pragma omp parallel for collapse(2) schedule(static)
        for (i64 n = 0; n < N; ++n)
            for (i64 c = 0; c < C; ++c) {
                double g = gamma ? gamma[c] : 1.0;
                for (i64 l = 0; l < L; ++l) {
                    i64 o = (n * C + c) * L + l;
                    dx[o] = dy[o] * g / sqrt(var[c] + eps);
                }
            }
    }
    if (dgamma || dbeta) {
#pragma omp parallel for schedule(static)
        for (i64 c = 0; c < C; ++c) {
            double sg = 0.0, sb = 0.0;
            for (i64 n = 0; n < N; ++n)
                for (i64 l = 0; l < L; ++l) {
                    i64 o = (n * C + c) * L + l;
                    if (dgamma) sg += dy[o] * (x[o] - mean[c]) / sqrt(var[c] + eps);
                    sb += dy[o];
                }
            if (dgamma) dgamma[c] = sg;
            if (dbeta) dbeta[c] = sb;
        }
    }
}

/* ---------------------------------------------------------------------------
 * Global average pool x[N,C,H,W] -> y[N,C] and its adjoint.
 * ------------------------------------------------------------------------- */
void orc_avgpool_forward(const double *x, double *y, i64 N, i64 C, i64 L)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 n = 0; n < N; ++n)
        for (i64 c = 0; c < C; ++c) {
            double acc = 0.0;
            for (i64 l = 0; l < L; ++l) acc += x[(n * C + c) * L + l];
            y[n * C + c] = acc / (double)L;
        }
}

void orc_avgpool_backward(const double *dy, double *dx, i64 N, i64 C, i64 L)
{
#pragma omp parallel for collapse(2) schedule(static)
    for (i64 n = 0; n < N; ++n)
        for (i64 c = 0; c < C; ++c)
            for (i64 l = 0; l < L; ++l) dx[(n * C + c) * L + l] = dy[n * C + c] / (double)L;
}

/* ---------------------------------------------------------------------------
 * Round float64 values once to a storage precision, in place:
 *   dtype 0: IEEE binary32, round to nearest even (the C conversion);
 *   dtype 1: bfloat16 (8 significant bits, binary32 exponent range), round
 *            to nearest even directly from the float64 value.
 * ------------------------------------------------------------------------- */
static double round_to_bf16(double v)
{
    if (!isfinite(v) || v == 0.0) return v;
    const double maxbf = ldexp(255.0, 120);     /* (2 - 2^-7) * 2^127 */
    int e;
    double m = frexp(fabs(v), &e);               /* |v| = m * 2^e, m in [0.5, 1) */
    int q = e - 8;                               /* quantum exponent for 8 significant bits */
    if (q < -133) q = -133;                      /* bf16 subnormal spacing is 2^-133 */
    (void)m;
    double r = nearbyint(ldexp(fabs(v), -q));    /* default rounding: ties to even */
    double out = ldexp(r, q);
    if (out > maxbf) out = INFINITY;
    return v < 0 ? -out : out;
}

void orc_round(double *a, i64 n, int dtype)
{
#pragma omp parallel for schedule(static)
    for (i64 i = 0; i < n; ++i)
        a[i] = dtype == 1 ? round_to_bf16(a[i]) : (double)(float)a[i];
}

/* Threads the OpenMP loops above use (reported with CPU timings). */
#ifdef _OPENMP
#include <omp.h>
#endif
int orc_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

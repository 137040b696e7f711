// Host runtime of libmemsave: argument validation, the save rule, saved-tensor
// records, the byte ledger and the C ABI declared in include/memsave.h.
//
// The save rule is Sec. 2.2.1 of the paper: for a layer that is linear in its
// input X and its weight W (and adds a bias b), the input Jacobian depends on
// W, the weight Jacobian on X and the bias Jacobian on nothing; the forward
// pass checks which of them require grad and keeps only what the Jacobians
// that backward will apply need.  BN in evaluation mode follows the same
// pattern with gamma as the weight (its input gradient needs gamma and the
// running variance, its gamma gradient needs x, the running mean and
// variance).  A transposed convolution is the adjoint of a convolution and
// keeps what a convolution keeps.  ReLU (Sec. 2.2.2) keeps one bit per
// element instead of its output, so the next linear layer's input is not
// kept alive by it; dropout (Sec. 2.2.2 too) keeps its generator's key and
// counter and draws the mask again in backward.
// Nothing in this file touches the device except through the
// launchers of device.h, and every check runs before the first launch.
#include <algorithm>
#include <initializer_list>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>

#include "../../include/memsave.h"
#include "../../include/memsave_testing.h"
#include "device.h"

namespace {

thread_local std::string g_err;

ms_status fail(ms_status s, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return s;
}

void clear_err() { g_err.clear(); }

// ------------------------------------------------------------------ ledger
std::atomic<uint64_t> g_live{0}, g_peak{0};
std::atomic<int64_t> g_records{0};

void ledger_add(uint64_t n) {
    uint64_t now = g_live.fetch_add(n) + n;
    uint64_t pk = g_peak.load();
    while (now > pk && !g_peak.compare_exchange_weak(pk, now)) {
    }
}

void ledger_sub(uint64_t n) { g_live.fetch_sub(n); }

// ------------------------------------------------------------------ tensors
constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;
constexpr uint32_t kMagic = 0x4d53524bu;  // "MSRK"

// Product of non-negative extents, saturated just above kMaxElems (the
// limit checks below must not be fooled by an int64 overflow).
int64_t capped_product(std::initializer_list<int64_t> f);

int64_t numel(const ms_tensor *t) {
    int64_t n = 1;
    for (int i = 0; i < t->ndim; ++i) n *= t->shape[i];
    return n;
}

size_t elt_size(int32_t dt) { return dt == MS_BF16 ? 2 : 4; }

int64_t capped_product(std::initializer_list<int64_t> f) {
    int64_t p = 1;
    for (int64_t v : f) {
        if (v == 0) return 0;
        if (p > (kMaxElems + 1) / v) p = kMaxElems + 1;
        else p = std::min<int64_t>(p * v, kMaxElems + 1);
    }
    return p;
}

bool dtype_ok(int32_t dt) { return dt == MS_F32 || dt == MS_BF16; }

// Basic sanity: ndim, non-negative extents, element limit, dtype.
ms_status check_tensor(const ms_tensor *t, const char *name, int ndim, bool need_data) {
    if (!t) return fail(MS_E_NULL, "%s is NULL", name);
    if (t->ndim != ndim) return fail(MS_E_SHAPE, "%s: expected %d dims, got %d", name, ndim, t->ndim);
    if (!dtype_ok(t->dtype)) return fail(MS_E_DTYPE, "%s: unsupported dtype %d", name, t->dtype);
    int64_t n = 1;
    for (int i = 0; i < ndim; ++i) {
        if (t->shape[i] < 0) return fail(MS_E_SHAPE, "%s: negative extent", name);
        if (t->shape[i] > kMaxElems) return fail(MS_E_UNSUPPORTED, "%s: extent too large", name);
        n *= t->shape[i];
        if (n > kMaxElems) return fail(MS_E_UNSUPPORTED, "%s: more than 2^31-1 elements", name);
    }
    if (need_data && n > 0 && t->data == nullptr) return fail(MS_E_NULL, "%s.data is NULL", name);
    return MS_OK;
}

// Channels-last 4-D: memory order N, H, W, C (dims of extent 1 may carry any stride).
bool is_nhwc(const ms_tensor *t) {
    if (numel(t) == 0) return true;   // no element is ever addressed
    const int64_t N = t->shape[0], C = t->shape[1], H = t->shape[2], W = t->shape[3];
    (void)N;
    const int64_t want[4] = {H * W * C, 1, W * C, C};
    for (int i = 0; i < 4; ++i)
        if (t->shape[i] > 1 && t->stride[i] != want[i]) return false;
    return true;
}

// Channels-last 5-D: memory order N, D, H, W, C.
bool is_ndhwc(const ms_tensor *t) {
    if (numel(t) == 0) return true;
    const int64_t C = t->shape[1], D = t->shape[2], H = t->shape[3], W = t->shape[4];
    const int64_t want[5] = {D * H * W * C, 1, H * W * C, W * C, C};
    for (int i = 0; i < 5; ++i)
        if (t->shape[i] > 1 && t->stride[i] != want[i]) return false;
    return true;
}

bool is_rowmajor2(const ms_tensor *t) {
    if (numel(t) == 0) return true;
    if (t->shape[1] > 1 && t->stride[1] != 1) return false;
    if (t->shape[0] > 1 && t->stride[0] != t->shape[1]) return false;
    return true;
}

bool is_contig1(const ms_tensor *t) { return t->shape[0] <= 1 || t->stride[0] == 1; }

// Any layout of an input: strides of the varying dims must be >= 0.
bool strides_ok(const ms_tensor *t) {
    for (int i = 0; i < t->ndim; ++i)
        if (t->shape[i] > 1 && t->stride[i] < 0) return false;
    return true;
}

// No two elements share an address: with the varying dims sorted by stride,
// each stride is at least the span of the faster ones (a strided sub-array
// of a dense array).  Outputs must satisfy this.
bool non_overlapping(const ms_tensor *t) {
    if (!strides_ok(t)) return false;
    if (numel(t) == 0) return true;
    int d[5], k = 0;
    for (int i = 0; i < t->ndim; ++i)
        if (t->shape[i] > 1) d[k++] = i;
    std::sort(d, d + k, [&](int a, int b) { return t->stride[a] < t->stride[b]; });
    int64_t span = 1;
    for (int i = 0; i < k; ++i) {
        if (t->stride[d[i]] < span) return false;
        span = t->stride[d[i]] * t->shape[d[i]];
    }
    return true;
}

// Every element of a dense block of numel(t) elements, in some order of the
// dims (channels-last, NCHW, a transposed matrix, ...).
bool dense_any_order(const ms_tensor *t) {
    if (!non_overlapping(t)) return false;
    if (numel(t) == 0) return true;
    int64_t lo_span = 1;
    int d[5], k = 0;
    for (int i = 0; i < t->ndim; ++i)
        if (t->shape[i] > 1) d[k++] = i;
    std::sort(d, d + k, [&](int a, int b) { return t->stride[a] < t->stride[b]; });
    for (int i = 0; i < k; ++i) {
        if (t->stride[d[i]] != lo_span) return false;
        lo_span *= t->shape[d[i]];
    }
    return true;
}

// Plain row-major [N, C, H, W] (PyTorch's default contiguous layout).
bool is_nchw(const ms_tensor *t) {
    if (t->ndim != 4) return false;
    const int64_t C = t->shape[1], H = t->shape[2], W = t->shape[3];
    const int64_t want[4] = {C * H * W, H * W, W, 1};
    for (int i = 0; i < 4; ++i)
        if (t->shape[i] > 1 && t->stride[i] != want[i]) return false;
    return true;
}

bool same_strides(const ms_tensor *a, const ms_tensor *b) {
    for (int i = 0; i < a->ndim; ++i)
        if (a->shape[i] > 1 && a->stride[i] != b->stride[i]) return false;
    return true;
}

// The dense layout the kernels read and write: channels-last for 4-D
// tensors (NHWC activations, KRSC filters), row-major for matrices.
bool canonical(const ms_tensor *t) {
    if (t->ndim == 4) return is_nhwc(t);
    if (t->ndim == 2) return is_rowmajor2(t);
    if (t->ndim == 5) return is_ndhwc(t);
    return is_contig1(t);
}

bool same_shape(const ms_tensor *a, const ms_tensor *b) {
    if (a->ndim != b->ndim) return false;
    for (int i = 0; i < a->ndim; ++i)
        if (a->shape[i] != b->shape[i]) return false;
    return true;
}

ms_tensor shape_only(const ms_tensor *t) {
    ms_tensor s = *t;
    s.data = nullptr;
    return s;
}

// ------------------------------------------------------------------ layer plan
struct Plan {
    int32_t kind = 0;
    int32_t dtype = 0;
    ms::ConvGeom g{};      // conv / linear; transposed conv: the convolution it is the adjoint of
    ms::Conv3dGeom q{};    // 3-D kinds: the (adjoint) 3-D convolution; g = q.g
    int64_t rows = 0;      // BN / avgpool: pixels; conv/linear bias grad rows
    int C = 0;             // BN / avgpool channels
    int L = 0;             // avgpool pixels per sample
    int Nb = 0;            // avgpool batch
    bool has_w = false, has_b = false;
    uint64_t x_bytes = 0, w_bytes = 0, stat_bytes = 0;
    int64_t n = 0;                           // ReLU / dropout: elements
    uint64_t bits_bytes = 0, y_bytes = 0;    // ReLU: 1-bit mask, output
    uint64_t mask8_bytes = 0;                // dropout: stock PyTorch's one-byte mask
    // layouts that are not the kernels' (staged through transient workspace)
    bool st_x = false, st_w = false, st_y = false;
    uint64_t out_bytes = 0;                  // bytes of y
    bool bn_nchw = false;                    // BN-eval on plain NCHW tensors: its sweeps run in place
    int64_t hw = 0;                          // BN-eval: H * W of a 4-D x
};

bool stageable(int32_t kind) {
    return kind == MS_CONV2D || kind == MS_CONV_TRANSPOSE2D || kind == MS_LINEAR || kind == MS_BN_EVAL ||
           kind == MS_AVGPOOL;
}

// Staging flags and the output size, once the kind's checks have passed.
void plan_layouts(Plan *pl, const ms_tensor *x, const ms_tensor *W, const ms_tensor *y) {
    if (!stageable(pl->kind)) return;
    pl->st_x = !canonical(x);
    pl->st_w = W && W->ndim >= 2 && !canonical(W);
    pl->st_y = y && !canonical(y);
    if (pl->kind == MS_BN_EVAL && x->ndim == 4) {
        pl->hw = x->shape[2] * x->shape[3];
        pl->bn_nchw = pl->st_x && is_nchw(x) && (!y || (pl->st_y && is_nchw(y)));
    }
    const uint64_t e = elt_size(pl->dtype);
    switch (pl->kind) {
    case MS_CONV2D: pl->out_bytes = (uint64_t)pl->g.N * pl->g.P * pl->g.Q * pl->g.K * e; break;
    case MS_CONV_TRANSPOSE2D: pl->out_bytes = (uint64_t)pl->g.N * pl->g.H * pl->g.W * pl->g.C * e; break;
    case MS_LINEAR: pl->out_bytes = (uint64_t)pl->g.N * pl->g.K * e; break;
    case MS_BN_EVAL: pl->out_bytes = pl->x_bytes; break;
    case MS_AVGPOOL: pl->out_bytes = (uint64_t)pl->Nb * pl->C * e; break;
    }
}

uint64_t relu_mask_bytes(int64_t n) { return n > 0 ? (uint64_t)((n + 31) / 32) * 4u : 0u; }


ms_status validate_forward_kind(const ms_layer *layer, const ms_tensor *x, const ms_tensor *W,
                                const ms_tensor *b, uint32_t mask, const ms_tensor *y, bool need_data,
                                Plan *pl);

ms_status validate_forward(const ms_layer *layer, const ms_tensor *x, const ms_tensor *W,
                           const ms_tensor *b, uint32_t mask, const ms_tensor *y, bool need_data,
                           Plan *pl) {
    const ms_status st = validate_forward_kind(layer, x, W, b, mask, y, need_data, pl);
    if (st == MS_OK) plan_layouts(pl, x, W, y);
    return st;
}

ms_status validate_forward_kind(const ms_layer *layer, const ms_tensor *x, const ms_tensor *W,
                                const ms_tensor *b, uint32_t mask, const ms_tensor *y, bool need_data,
                                Plan *pl) {
    if (!layer) return fail(MS_E_NULL, "layer is NULL");
    if (mask & ~7u) return fail(MS_E_MASK, "mask 0x%x has bits outside INPUT|WEIGHT|BIAS", mask);
    pl->kind = layer->kind;
    pl->has_w = W != nullptr;
    pl->has_b = b != nullptr;
    if ((mask & MS_RG_WEIGHT) && !W) return fail(MS_E_MASK, "WEIGHT bit set but the layer has no weight");
    if ((mask & MS_RG_BIAS) && !b) return fail(MS_E_MASK, "BIAS bit set but the layer has no bias");
    ms_status st;
    switch (layer->kind) {
    case MS_CONV2D: {
        if ((st = check_tensor(x, "x", 4, need_data))) return st;
        if (!W) return fail(MS_E_NULL, "conv2d needs W");
        if ((st = check_tensor(W, "W", 4, need_data))) return st;
        if (x->dtype != W->dtype) return fail(MS_E_DTYPE, "x and W dtypes differ");
        if (!strides_ok(x) || !strides_ok(W)) return fail(MS_E_LAYOUT, "x and W need non-negative strides");
        const int64_t N = x->shape[0], C = x->shape[1], H = x->shape[2], Wd = x->shape[3];
        const int64_t K = W->shape[0], R = W->shape[2], S = W->shape[3];
        if (W->shape[1] != C) return fail(MS_E_SHAPE, "W has %lld input channels, x has %lld",
                                          (long long)W->shape[1], (long long)C);
        if (layer->stride[0] < 1 || layer->stride[1] < 1) return fail(MS_E_ARG, "stride must be >= 1");
        if (layer->pad[0] < 0 || layer->pad[1] < 0) return fail(MS_E_ARG, "pad must be >= 0");
        if (C < 1 || K < 1 || R < 1 || S < 1 || H < 1 || Wd < 1)
            return fail(MS_E_SHAPE, "conv2d extents C, K, R, S, H, W must be >= 1");
        const int64_t Hp = H + 2 * (int64_t)layer->pad[0], Wp = Wd + 2 * (int64_t)layer->pad[1];
        if (Hp < R || Wp < S) return fail(MS_E_SHAPE, "kernel larger than the padded input");
        if (Hp > kMaxElems || Wp > kMaxElems) return fail(MS_E_UNSUPPORTED, "padding too large");
        const int64_t P = (Hp - R) / layer->stride[0] + 1, Q = (Wp - S) / layer->stride[1] + 1;
        if (b) {
            if ((st = check_tensor(b, "b", 1, need_data))) return st;
            if (b->dtype != x->dtype) return fail(MS_E_DTYPE, "b dtype differs from x");
            if (b->shape[0] != K) return fail(MS_E_SHAPE, "b must have K elements");
            if (!is_contig1(b)) return fail(MS_E_LAYOUT, "b must be contiguous");
        }
        if (y) {
            if ((st = check_tensor(y, "y", 4, need_data))) return st;
            if (y->dtype != x->dtype) return fail(MS_E_DTYPE, "y dtype differs from x");
            if (y->shape[0] != N || y->shape[1] != K || y->shape[2] != P || y->shape[3] != Q)
                return fail(MS_E_SHAPE, "y must be [%lld,%lld,%lld,%lld]", (long long)N, (long long)K,
                            (long long)P, (long long)Q);
            if (!non_overlapping(y)) return fail(MS_E_LAYOUT, "y must not overlap itself");
        }
        pl->dtype = x->dtype;
        pl->g = ms::ConvGeom{(int)N, (int)C, (int)H, (int)Wd, (int)K, (int)R, (int)S, (int)P, (int)Q,
                             layer->stride[0], layer->stride[1], layer->pad[0], layer->pad[1]};
        if (capped_product({N, P, Q, K}) > kMaxElems) return fail(MS_E_UNSUPPORTED, "output has more than 2^31-1 elements");
        pl->rows = N * P * Q;
        pl->x_bytes = (uint64_t)numel(x) * elt_size(x->dtype);
        pl->w_bytes = (uint64_t)numel(W) * elt_size(W->dtype);
        return MS_OK;
    }
    case MS_CONV_TRANSPOSE2D: {
        if ((st = check_tensor(x, "x", 4, need_data))) return st;
        if (!W) return fail(MS_E_NULL, "conv_transpose2d needs W");
        if ((st = check_tensor(W, "W", 4, need_data))) return st;
        if (x->dtype != W->dtype) return fail(MS_E_DTYPE, "x and W dtypes differ");
        if (!strides_ok(x) || !strides_ok(W)) return fail(MS_E_LAYOUT, "x and W need non-negative strides");
        const int64_t N = x->shape[0], Ci = x->shape[1], H = x->shape[2], Wd = x->shape[3];
        const int64_t Co = W->shape[1], R = W->shape[2], S = W->shape[3];
        if (W->shape[0] != Ci) return fail(MS_E_SHAPE, "W has %lld input channels, x has %lld",
                                           (long long)W->shape[0], (long long)Ci);
        if (layer->stride[0] < 1 || layer->stride[1] < 1) return fail(MS_E_ARG, "stride must be >= 1");
        if (layer->pad[0] < 0 || layer->pad[1] < 0) return fail(MS_E_ARG, "pad must be >= 0");
        for (int i = 0; i < 2; ++i)
            if (layer->out_pad[i] < 0 || layer->out_pad[i] >= layer->stride[i])
                return fail(MS_E_ARG, "out_pad must satisfy 0 <= out_pad < stride");
        if (Ci < 1 || Co < 1 || R < 1 || S < 1 || H < 1 || Wd < 1)
            return fail(MS_E_SHAPE, "conv_transpose2d extents C_in, C_out, R, S, H, W must be >= 1");
        const int64_t Ho = (H - 1) * layer->stride[0] - 2 * (int64_t)layer->pad[0] + R + layer->out_pad[0];
        const int64_t Wo = (Wd - 1) * layer->stride[1] - 2 * (int64_t)layer->pad[1] + S + layer->out_pad[1];
        if (Ho < 1 || Wo < 1) return fail(MS_E_SHAPE, "output would be empty");
        if (Ho + 2 * (int64_t)layer->pad[0] > kMaxElems || Wo + 2 * (int64_t)layer->pad[1] > kMaxElems)
            return fail(MS_E_UNSUPPORTED, "output extent too large");
        if (b) {
            if ((st = check_tensor(b, "b", 1, need_data))) return st;
            if (b->dtype != x->dtype) return fail(MS_E_DTYPE, "b dtype differs from x");
            if (b->shape[0] != Co) return fail(MS_E_SHAPE, "b must have C_out elements");
            if (!is_contig1(b)) return fail(MS_E_LAYOUT, "b must be contiguous");
        }
        if (y) {
            if ((st = check_tensor(y, "y", 4, need_data))) return st;
            if (y->dtype != x->dtype) return fail(MS_E_DTYPE, "y dtype differs from x");
            if (y->shape[0] != N || y->shape[1] != Co || y->shape[2] != Ho || y->shape[3] != Wo)
                return fail(MS_E_SHAPE, "y must be [%lld,%lld,%lld,%lld]", (long long)N, (long long)Co,
                            (long long)Ho, (long long)Wo);
            if (!non_overlapping(y)) return fail(MS_E_LAYOUT, "y must not overlap itself");
        }
        if (capped_product({N, Ho, Wo, Co}) > kMaxElems)
            return fail(MS_E_UNSUPPORTED, "output has more than 2^31-1 elements");
        pl->dtype = x->dtype;
        // the convolution y -> x with filter W: input [N,C_out,H_out,W_out], K = C_in filters,
        // output [N,C_in,H,W]; out_pad < stride makes its output extent exactly H x W
        pl->g = ms::ConvGeom{(int)N, (int)Co, (int)Ho, (int)Wo, (int)Ci, (int)R, (int)S, (int)H, (int)Wd,
                             layer->stride[0], layer->stride[1], layer->pad[0], layer->pad[1]};
        if ((Ho + 2 * layer->pad[0] - R) / layer->stride[0] + 1 != H ||
            (Wo + 2 * layer->pad[1] - S) / layer->stride[1] + 1 != Wd)
            return fail(MS_E_ARG, "inconsistent transposed-convolution geometry");
        pl->rows = N * Ho * Wo;
        pl->x_bytes = (uint64_t)numel(x) * elt_size(x->dtype);
        pl->w_bytes = (uint64_t)numel(W) * elt_size(W->dtype);
        return MS_OK;
    }
    case MS_CONV3D:
    case MS_CONV_TRANSPOSE3D: {
        const bool tr = layer->kind == MS_CONV_TRANSPOSE3D;
        if ((st = check_tensor(x, "x", 5, need_data))) return st;
        if (!W) return fail(MS_E_NULL, "3-D convolution needs W");
        if ((st = check_tensor(W, "W", 5, need_data))) return st;
        if (x->dtype != W->dtype) return fail(MS_E_DTYPE, "x and W dtypes differ");
        if (!is_ndhwc(x)) return fail(MS_E_LAYOUT, "x must be channels-last (NDHWC)");
        if (!is_ndhwc(W)) return fail(MS_E_LAYOUT, "W must be channels-last (memory [W0][T][R][S][W1])");
        const int64_t N = x->shape[0], Cx = x->shape[1], D = x->shape[2], H = x->shape[3], Wd = x->shape[4];
        const int64_t T = W->shape[2], R = W->shape[3], S = W->shape[4];
        const int64_t Cw = tr ? W->shape[0] : W->shape[1];   // W's extent that must match x's channels
        const int64_t Cy = tr ? W->shape[1] : W->shape[0];   // output channels
        if (Cw != Cx) return fail(MS_E_SHAPE, "W has %lld input channels, x has %lld", (long long)Cw, (long long)Cx);
        const int32_t sd = layer->stride_d, pd = layer->pad_d, od = layer->out_pad_d;
        if (layer->stride[0] < 1 || layer->stride[1] < 1 || sd < 1) return fail(MS_E_ARG, "stride must be >= 1");
        if (layer->pad[0] < 0 || layer->pad[1] < 0 || pd < 0) return fail(MS_E_ARG, "pad must be >= 0");
        if (tr && (od < 0 || od >= sd || layer->out_pad[0] < 0 || layer->out_pad[0] >= layer->stride[0] ||
                   layer->out_pad[1] < 0 || layer->out_pad[1] >= layer->stride[1]))
            return fail(MS_E_ARG, "out_pad must satisfy 0 <= out_pad < stride");
        if (Cx < 1 || Cy < 1 || T < 1 || R < 1 || S < 1 || D < 1 || H < 1 || Wd < 1)
            return fail(MS_E_SHAPE, "3-D convolution extents must be >= 1");
        int64_t o[3];
        const int64_t in[3] = {D, H, Wd}, k[3] = {T, R, S};
        const int64_t sv[3] = {sd, layer->stride[0], layer->stride[1]}, pv[3] = {pd, layer->pad[0], layer->pad[1]};
        const int64_t ov[3] = {od, layer->out_pad[0], layer->out_pad[1]};
        for (int i = 0; i < 3; ++i) {
            if (in[i] + 2 * pv[i] > kMaxElems) return fail(MS_E_UNSUPPORTED, "padding too large");
            if (tr) {
                o[i] = (in[i] - 1) * sv[i] - 2 * pv[i] + k[i] + ov[i];
                if (o[i] < 1) return fail(MS_E_SHAPE, "output would be empty");
                if (o[i] + 2 * pv[i] > kMaxElems) return fail(MS_E_UNSUPPORTED, "output extent too large");
            } else {
                if (in[i] + 2 * pv[i] < k[i]) return fail(MS_E_SHAPE, "kernel larger than the padded input");
                o[i] = (in[i] + 2 * pv[i] - k[i]) / sv[i] + 1;
            }
        }
        if (b) {
            if ((st = check_tensor(b, "b", 1, need_data))) return st;
            if (b->dtype != x->dtype) return fail(MS_E_DTYPE, "b dtype differs from x");
            if (b->shape[0] != Cy) return fail(MS_E_SHAPE, "b must have %lld elements", (long long)Cy);
            if (!is_contig1(b)) return fail(MS_E_LAYOUT, "b must be contiguous");
        }
        if (y) {
            if ((st = check_tensor(y, "y", 5, need_data))) return st;
            if (y->dtype != x->dtype) return fail(MS_E_DTYPE, "y dtype differs from x");
            if (y->shape[0] != N || y->shape[1] != Cy || y->shape[2] != o[0] || y->shape[3] != o[1] ||
                y->shape[4] != o[2])
                return fail(MS_E_SHAPE, "y must be [%lld,%lld,%lld,%lld,%lld]", (long long)N, (long long)Cy,
                            (long long)o[0], (long long)o[1], (long long)o[2]);
            if (!is_ndhwc(y)) return fail(MS_E_LAYOUT, "y must be channels-last (NDHWC)");
        }
        if (capped_product({N, o[0], o[1], o[2], Cy}) > kMaxElems)
            return fail(MS_E_UNSUPPORTED, "output has more than 2^31-1 elements");
        // the 3-D convolution u -> v this layer runs (itself, or the one it is the adjoint of)
        const int64_t Cu = tr ? Cy : Cx, Cv = tr ? Cx : Cy;
        const int64_t *du = tr ? o : in, *dv = tr ? in : o;
        const int64_t folded = capped_product({N, dv[0], du[1], du[2], T, Cu});   // [N*Dv][Hu][Wu][T*Cu]
        if (folded > kMaxElems || T * Cu > kMaxElems || N * dv[0] > kMaxElems)
            return fail(MS_E_UNSUPPORTED, "depth-folded input has more than 2^31-1 elements");
        pl->dtype = x->dtype;
        pl->q.N = (int)N;
        pl->q.C = (int)Cu;
        pl->q.Din = (int)du[0];
        pl->q.Do = (int)dv[0];
        pl->q.T = (int)T;
        pl->q.sd = sd;
        pl->q.pd = pd;
        pl->q.g = ms::ConvGeom{(int)(N * dv[0]), (int)(T * Cu), (int)du[1], (int)du[2], (int)Cv, (int)R, (int)S,
                               (int)dv[1], (int)dv[2], layer->stride[0], layer->stride[1], layer->pad[0], layer->pad[1]};
        if ((du[1] + 2 * layer->pad[0] - R) / layer->stride[0] + 1 != dv[1] ||
            (du[2] + 2 * layer->pad[1] - S) / layer->stride[1] + 1 != dv[2] || (du[0] + 2 * pd - T) / sd + 1 != dv[0])
            return fail(MS_E_ARG, "inconsistent 3-D convolution geometry");
        pl->g = pl->q.g;
        pl->rows = N * o[0] * o[1] * o[2];   // bias-gradient rows of the output
        pl->C = (int)Cy;
        pl->x_bytes = (uint64_t)numel(x) * elt_size(x->dtype);
        pl->w_bytes = (uint64_t)numel(W) * elt_size(W->dtype);
        return MS_OK;
    }
    case MS_LINEAR: {
        if ((st = check_tensor(x, "x", 2, need_data))) return st;
        if (!W) return fail(MS_E_NULL, "linear needs W");
        if ((st = check_tensor(W, "W", 2, need_data))) return st;
        if (x->dtype != W->dtype) return fail(MS_E_DTYPE, "x and W dtypes differ");
        if (!strides_ok(x) || !strides_ok(W)) return fail(MS_E_LAYOUT, "x and W need non-negative strides");
        const int64_t M = x->shape[0], Kin = x->shape[1], Nout = W->shape[0];
        if (W->shape[1] != Kin) return fail(MS_E_SHAPE, "W has %lld input features, x has %lld",
                                            (long long)W->shape[1], (long long)Kin);
        if (b) {
            if ((st = check_tensor(b, "b", 1, need_data))) return st;
            if (b->dtype != x->dtype) return fail(MS_E_DTYPE, "b dtype differs from x");
            if (b->shape[0] != Nout) return fail(MS_E_SHAPE, "b must have N_out elements");
            if (!is_contig1(b)) return fail(MS_E_LAYOUT, "b must be contiguous");
        }
        if (y) {
            if ((st = check_tensor(y, "y", 2, need_data))) return st;
            if (y->dtype != x->dtype) return fail(MS_E_DTYPE, "y dtype differs from x");
            if (y->shape[0] != M || y->shape[1] != Nout) return fail(MS_E_SHAPE, "y must be [M, N_out]");
            if (!non_overlapping(y)) return fail(MS_E_LAYOUT, "y must not overlap itself");
        }
        pl->dtype = x->dtype;
        pl->g = ms::ConvGeom{(int)M, (int)Kin, 1, 1, (int)Nout, 1, 1, 1, 1, 1, 1, 0, 0};
        pl->rows = M;
        pl->x_bytes = (uint64_t)numel(x) * elt_size(x->dtype);
        pl->w_bytes = (uint64_t)numel(W) * elt_size(W->dtype);
        return MS_OK;
    }
    case MS_BN_EVAL: {
        if (!x) return fail(MS_E_NULL, "x is NULL");
        const int nd = x->ndim;
        if (nd != 2 && nd != 4) return fail(MS_E_SHAPE, "BN-eval x must be [N,C] or [N,C,H,W]");
        if ((st = check_tensor(x, "x", nd, need_data))) return st;
        if (!strides_ok(x)) return fail(MS_E_LAYOUT, "x needs non-negative strides");
        const int64_t C = x->shape[1];
        if (C < 1) return fail(MS_E_SHAPE, "BN-eval needs C >= 1");
        const ms_tensor *mean = layer->running_mean, *var = layer->running_var;
        if (!mean || !var) return fail(MS_E_NULL, "BN-eval needs running_mean and running_var");
        if ((st = check_tensor(mean, "running_mean", 1, need_data))) return st;
        if ((st = check_tensor(var, "running_var", 1, need_data))) return st;
        const ms_tensor *ps[4] = {W, b, mean, var};
        const char *nm[4] = {"W (gamma)", "b (beta)", "running_mean", "running_var"};
        for (int i = 0; i < 4; ++i) {
            if (!ps[i]) continue;
            if (i < 2 && (st = check_tensor(ps[i], nm[i], 1, need_data))) return st;
            if (ps[i]->dtype != x->dtype) return fail(MS_E_DTYPE, "%s dtype differs from x", nm[i]);
            if (ps[i]->shape[0] != C) return fail(MS_E_SHAPE, "%s must have C elements", nm[i]);
            if (!is_contig1(ps[i])) return fail(MS_E_LAYOUT, "%s must be contiguous", nm[i]);
        }
        if (!(layer->eps >= 0.f) || !std::isfinite(layer->eps)) return fail(MS_E_ARG, "eps must be finite and >= 0");
        if (y) {
            if ((st = check_tensor(y, "y", nd, need_data))) return st;
            if (y->dtype != x->dtype) return fail(MS_E_DTYPE, "y dtype differs from x");
            if (!same_shape(x, y)) return fail(MS_E_SHAPE, "y must have the shape of x");
            if (!non_overlapping(y)) return fail(MS_E_LAYOUT, "y must not overlap itself");
        }
        pl->dtype = x->dtype;
        pl->C = (int)C;
        pl->rows = C > 0 ? numel(x) / C : 0;
        pl->x_bytes = (uint64_t)numel(x) * elt_size(x->dtype);
        pl->w_bytes = W ? (uint64_t)C * elt_size(x->dtype) : 0;
        pl->stat_bytes = (uint64_t)C * elt_size(x->dtype);
        return MS_OK;
    }
    case MS_AVGPOOL: {
        if (W || b) return fail(MS_E_ARG, "avgpool takes no W or b");
        if (mask & ~(uint32_t)MS_RG_INPUT) return fail(MS_E_MASK, "avgpool has no parameters");
        if ((st = check_tensor(x, "x", 4, need_data))) return st;
        if (!strides_ok(x)) return fail(MS_E_LAYOUT, "x needs non-negative strides");
        const int64_t N = x->shape[0], C = x->shape[1], L = x->shape[2] * x->shape[3];
        if (C < 1 || L < 1) return fail(MS_E_SHAPE, "avgpool needs C, H, W >= 1");
        if (y) {
            if ((st = check_tensor(y, "y", 2, need_data))) return st;
            if (y->dtype != x->dtype) return fail(MS_E_DTYPE, "y dtype differs from x");
            if (y->shape[0] != N || y->shape[1] != C) return fail(MS_E_SHAPE, "y must be [N, C]");
            if (!non_overlapping(y)) return fail(MS_E_LAYOUT, "y must not overlap itself");
        }
        pl->dtype = x->dtype;
        pl->C = (int)C;
        pl->L = (int)L;
        pl->Nb = (int)N;
        pl->rows = N * L;
        pl->x_bytes = (uint64_t)numel(x) * elt_size(x->dtype);
        return MS_OK;
    }
    case MS_RELU:
    case MS_DROPOUT: {
        const char *nm = layer->kind == MS_RELU ? "ReLU" : "dropout";
        if (W || b) return fail(MS_E_ARG, "%s takes no W or b", nm);
        if (mask & ~(uint32_t)MS_RG_INPUT) return fail(MS_E_MASK, "%s has no parameters", nm);
        if (!x) return fail(MS_E_NULL, "x is NULL");
        const int nd = x->ndim;
        if (nd != 1 && nd != 2 && nd != 4) return fail(MS_E_SHAPE, "%s x must have 1, 2 or 4 dims", nm);
        if ((st = check_tensor(x, "x", nd, need_data))) return st;
        if (!dense_any_order(x)) return fail(MS_E_LAYOUT, "x must be dense (any order of its dims)");
        if (y) {
            if ((st = check_tensor(y, "y", nd, need_data))) return st;
            if (y->dtype != x->dtype) return fail(MS_E_DTYPE, "y dtype differs from x");
            if (!same_shape(x, y)) return fail(MS_E_SHAPE, "y must have the shape of x");
            if (!dense_any_order(y) || !same_strides(x, y)) return fail(MS_E_LAYOUT, "y must be in the layout of x");
        }
        pl->dtype = x->dtype;
        pl->n = numel(x);
        pl->x_bytes = (uint64_t)pl->n * elt_size(x->dtype);
        pl->y_bytes = pl->x_bytes;
        pl->bits_bytes = relu_mask_bytes(pl->n);
        pl->mask8_bytes = (uint64_t)pl->n;
        return MS_OK;
    }
    default:
        return fail(MS_E_ARG, "unknown layer kind %d", layer->kind);
    }
}

// The save rule.  Returns MS_SAVED_* bits for `mask` under `policy`.
uint32_t borrowed_bits(int32_t kind, uint32_t mask, int32_t policy, bool has_w, bool has_b) {
    if (policy == MS_POLICY_ALL_TRUE)
        mask = MS_RG_INPUT | (has_w ? (uint32_t)MS_RG_WEIGHT : 0u) | (has_b ? (uint32_t)MS_RG_BIAS : 0u);
    if (mask == 0) return 0;
    const bool in = mask & MS_RG_INPUT, w = mask & MS_RG_WEIGHT;
    switch (kind) {
    case MS_CONV2D:
    case MS_CONV_TRANSPOSE2D:   // stock PyTorch keeps both for either (Fig. 2, App. B)
    case MS_CONV3D:
    case MS_CONV_TRANSPOSE3D:
        if (policy == MS_POLICY_PYTORCH_DEFAULT) return MS_SAVED_X | MS_SAVED_W;
        return (w ? (uint32_t)MS_SAVED_X : 0u) | (in ? (uint32_t)MS_SAVED_W : 0u);
    case MS_LINEAR:   // PyTorch's Linear is already selective (App. B)
        return (w ? (uint32_t)MS_SAVED_X : 0u) | (in ? (uint32_t)MS_SAVED_W : 0u);
    case MS_BN_EVAL:
        if (policy == MS_POLICY_PYTORCH_DEFAULT)
            return MS_SAVED_X | (has_w ? (uint32_t)MS_SAVED_W : 0u) | MS_SAVED_MEAN | MS_SAVED_VAR;
        return (w ? (uint32_t)(MS_SAVED_X | MS_SAVED_MEAN) : 0u) | (in && has_w ? (uint32_t)MS_SAVED_W : 0u) |
               ((in || w) ? (uint32_t)MS_SAVED_VAR : 0u);
    case MS_RELU:   // stock PyTorch keeps the output; this library one bit per element
        if (!in) return 0;
        return policy == MS_POLICY_PYTORCH_DEFAULT ? (uint32_t)MS_SAVED_Y : (uint32_t)MS_SAVED_BITS;
    case MS_DROPOUT:   // stock PyTorch keeps a one-byte mask; this library the generator state
        return in && policy == MS_POLICY_PYTORCH_DEFAULT ? (uint32_t)MS_SAVED_MASK8 : 0u;
    default:
        return 0;
    }
}

uint32_t kernel_bits(int32_t kind, uint32_t mask) {
    uint32_t k = 0;
    if (mask & MS_RG_INPUT) k |= MS_K_DGRAD;
    if (kind != MS_AVGPOOL) {
        if (mask & MS_RG_WEIGHT) k |= MS_K_WGRAD;
        if (mask & MS_RG_BIAS) k |= MS_K_BGRAD;
    }
    return k;
}

size_t backward_workspace(const Plan &pl, uint32_t kernels) {
    size_t ws = 0;
    if (pl.kind == MS_CONV2D || pl.kind == MS_LINEAR) {
        // without a weight gradient, the bias gradient may ride on the input gradient
        if (kernels & MS_K_DGRAD)
            ws = std::max(ws, ms::conv_dgrad_workspace(pl.dtype, pl.g,
                                                       (kernels & MS_K_BGRAD) && !(kernels & MS_K_WGRAD)));
        if (kernels & MS_K_WGRAD)
            ws = std::max(ws, ms::conv_wgrad_workspace(pl.dtype, pl.g, (kernels & MS_K_BGRAD) != 0));
        if (kernels & MS_K_BGRAD) ws = std::max(ws, ms::colsum_workspace(pl.dtype, pl.rows, pl.g.K));
    } else if (pl.kind == MS_CONV_TRANSPOSE2D) {
        if (kernels & MS_K_DGRAD) ws = std::max(ws, ms::conv_fwd_workspace(pl.dtype, pl.g));
        if (kernels & MS_K_WGRAD) ws = std::max(ws, ms::conv_wgrad_workspace(pl.dtype, pl.g, false));
        if (kernels & MS_K_BGRAD) ws = std::max(ws, ms::colsum_workspace(pl.dtype, pl.rows, pl.g.C));
    } else if (pl.kind == MS_CONV3D) {
        if (kernels & MS_K_DGRAD) ws = std::max(ws, ms::conv3d_dgrad_workspace(pl.dtype, pl.q));
        if (kernels & MS_K_WGRAD)
            ws = std::max(ws, ms::conv3d_wgrad_workspace(pl.dtype, pl.q, (kernels & MS_K_BGRAD) != 0));
        if (kernels & MS_K_BGRAD) ws = std::max(ws, ms::colsum_workspace(pl.dtype, pl.rows, pl.C));
    } else if (pl.kind == MS_CONV_TRANSPOSE3D) {
        if (kernels & MS_K_DGRAD) ws = std::max(ws, ms::conv3d_fwd_workspace(pl.dtype, pl.q));
        if (kernels & MS_K_WGRAD) ws = std::max(ws, ms::conv3d_wgrad_workspace(pl.dtype, pl.q, false));
        if (kernels & MS_K_BGRAD) ws = std::max(ws, ms::colsum_workspace(pl.dtype, pl.rows, pl.C));
    } else if (pl.kind == MS_BN_EVAL) {
        if (kernels & (MS_K_WGRAD | MS_K_BGRAD)) ws = ms::bn_bwd_workspace(pl.dtype, pl.rows, pl.C);
    }
    return ws;
}

uint64_t backward_staging(const Plan &pl, uint32_t kernels);

ms_account make_account(const Plan &pl, uint32_t mask, uint32_t borrowed, uint32_t kernels) {
    ms_account a{};
    a.mask = mask;
    a.borrowed = borrowed;
    a.kernels = kernels;
    a.saved_activation_bytes = ((borrowed & MS_SAVED_X) ? pl.x_bytes : 0) +
                               ((borrowed & MS_SAVED_BITS) ? pl.bits_bytes : 0) +
                               ((borrowed & MS_SAVED_Y) ? pl.y_bytes : 0) +
                               ((borrowed & MS_SAVED_MASK8) ? pl.mask8_bytes : 0);
    uint64_t pb = 0;
    if (borrowed & MS_SAVED_W) pb += pl.w_bytes;
    if (borrowed & MS_SAVED_MEAN) pb += pl.stat_bytes;
    if (borrowed & MS_SAVED_VAR) pb += pl.stat_bytes;
    a.referenced_param_bytes = pb;
    a.transient_workspace_bytes = backward_workspace(pl, kernels) + backward_staging(pl, kernels);
    return a;
}

ms_status hip_fail(int err, const char *what) {
    return fail(MS_E_HIP, "%s failed with HIP error %d", what, err);
}

// ------------------------------------------------------------------ layout staging
// A caller tensor that is not in the kernels' layout (NCHW, a strided
// slice, a transposed matrix) is copied into a dense channels-last (or
// row-major) stand-in in transient workspace before the launch, and an
// output is written to such a stand-in and copied out after it.  The record
// still borrows the caller's own tensor.
constexpr size_t kNoStage = ~size_t(0);

size_t al256(size_t n) { return (n + 255) / 256 * 256; }

struct Stager {
    size_t bytes = 0;
    // Offset of t's stand-in, or kNoStage when t is used in place.
    size_t add(const ms_tensor *t) {
        if (!t || !t->data || numel(t) == 0 || canonical(t)) return kNoStage;
        const size_t off = bytes;
        bytes += al256((size_t)numel(t) * elt_size(t->dtype));
        return off;
    }
};

// The copy between t's layout and its dense stand-in, over (n, h, w, c) for
// 4-D tensors and (m, -, -, k) for matrices.
void copy_desc(const ms_tensor *t, int64_t ext[4], int64_t s[4], int64_t dense[4]) {
    if (t->ndim == 4) {
        const int64_t N = t->shape[0], C = t->shape[1], H = t->shape[2], W = t->shape[3];
        const int64_t e[4] = {N, H, W, C}, st[4] = {t->stride[0], t->stride[2], t->stride[3], t->stride[1]},
                      d[4] = {H * W * C, W * C, C, 1};
        for (int i = 0; i < 4; ++i) ext[i] = e[i], s[i] = st[i], dense[i] = d[i];
    } else {
        const int64_t e[4] = {t->shape[0], 1, 1, t->shape[1]}, st[4] = {t->stride[0], 0, 0, t->stride[1]},
                      d[4] = {t->shape[1], 0, 0, 1};
        for (int i = 0; i < 4; ++i) ext[i] = e[i], s[i] = st[i], dense[i] = d[i];
    }
}

int stage_in(const ms_tensor *t, char *base, size_t off, void *stream) {
    if (off == kNoStage) return 0;
    int64_t ext[4], s[4], d[4];
    copy_desc(t, ext, s, d);
    return ms::launch_copy4(t->dtype, t->data, ext, s, base + off, d, stream);
}

int stage_out(const ms_tensor *t, char *base, size_t off, void *stream) {
    if (off == kNoStage) return 0;
    int64_t ext[4], s[4], d[4];
    copy_desc(t, ext, s, d);
    return ms::launch_copy4(t->dtype, base + off, ext, d, t->data, s, stream);
}

// Data pointer the kernels use for t: its stand-in or the caller's memory.
void *kptr(const ms_tensor *t, char *base, size_t off) {
    if (!t) return nullptr;
    return off == kNoStage ? t->data : base + off;
}

// Staging bytes a backward with `kernels` needs, taking the output
// gradient in y's layout and the input and weight gradients in x's and W's.
uint64_t backward_staging(const Plan &pl, uint32_t kernels) {
    if (!stageable(pl.kind)) return 0;
    if (pl.bn_nchw && kernels == MS_K_DGRAD) return 0;   // dx alone: the in-place NCHW sweep
    const bool wg = kernels & MS_K_WGRAD, dg = kernels & MS_K_DGRAD;
    uint64_t b = pl.st_y ? al256(pl.out_bytes) : 0;               // grad_y
    if (pl.st_x && wg && pl.kind != MS_AVGPOOL) b += al256(pl.x_bytes);   // x read by the weight gradient
    if (pl.st_w && dg) b += al256(pl.w_bytes);                      // W read by the input gradient
    if (pl.st_x && dg) b += al256(pl.x_bytes);                      // grad_x
    if (pl.st_w && wg) b += al256(pl.w_bytes);                      // grad_W
    return b;
}

}  // namespace

struct ms_record {
    uint32_t magic;
    Plan plan;
    float eps;
    ms_tensor x, W, b, mean, var, y;   // data non-NULL only for borrowed tensors
    void *bits;                         // ReLU: the borrowed 1-bit mask
    uint64_t seed, offset;              // dropout: generator key and first block
    uint32_t thresh;                    // dropout: keep iff word >= thresh
    float scale;                        // dropout: 1 / (1 - p) (0 when p = 1)
    int drop_all;                       // dropout: p = 1
    ms_account acct;
    bool consumed;
    bool released;
};

namespace {

void release(ms_record *r) {
    if (!r->released) {
        ledger_sub(r->acct.saved_activation_bytes);
        r->released = true;
        r->x.data = nullptr;
        r->W.data = nullptr;
        r->mean.data = nullptr;
        r->var.data = nullptr;
        r->bits = nullptr;
    }
}

ms_status check_grad(const ms_tensor *g, const ms_tensor *primal, const char *name, int32_t kind, bool output) {
    ms_status st = check_tensor(g, name, primal->ndim, true);
    if (st) return st;
    if (g->dtype != primal->dtype) return fail(MS_E_DTYPE, "%s dtype must match its primal", name);
    if (!same_shape(g, primal)) return fail(MS_E_SHAPE, "%s shape must match its primal", name);
    if (g->ndim == 5 && !is_ndhwc(g)) return fail(MS_E_LAYOUT, "%s must be channels-last", name);
    if (g->ndim == 1 && !is_contig1(g)) return fail(MS_E_LAYOUT, "%s must be contiguous", name);
    if (kind == MS_RELU || kind == MS_DROPOUT) {
        // elementwise in memory order: the layout of the forward's tensors
        if (!dense_any_order(g) || !same_strides(g, primal)) return fail(MS_E_LAYOUT, "%s must be in the layout of x", name);
    } else if (output ? !non_overlapping(g) : !strides_ok(g)) {
        return fail(MS_E_LAYOUT, output ? "%s must not overlap itself" : "%s needs non-negative strides", name);
    }
    return MS_OK;
}

}  // namespace

extern "C" {

ms_status ms_layer_forward(const ms_layer *layer, const ms_tensor *x, const ms_tensor *W,
                           const ms_tensor *b, uint32_t mask, const ms_tensor *y, ms_record **rec,
                           void *stream) {
    clear_err();
    if (!rec) return fail(MS_E_NULL, "rec is NULL");
    *rec = nullptr;
    if (!y) return fail(MS_E_NULL, "y is NULL");
    if (layer && layer->kind == MS_RELU) return fail(MS_E_ARG, "ReLU runs through ms_relu_forward()");
    if (layer && layer->kind == MS_DROPOUT) return fail(MS_E_ARG, "dropout runs through ms_dropout_forward()");
    Plan pl;
    ms_status st = validate_forward(layer, x, W, b, mask, y, true, &pl);
    if (st) return st;
    const uint32_t borrowed = borrowed_bits(pl.kind, mask, MS_POLICY_SELECTIVE, pl.has_w, pl.has_b);
    const uint32_t kernels = kernel_bits(pl.kind, mask);
    // transient forward workspace: stand-ins of tensors in other layouts,
    // then the kernels' own (zero-padded channel copies for channel counts
    // that are not a multiple of 8), taken before anything is launched
    Stager sg;
    const bool stg = stageable(pl.kind) && !pl.bn_nchw;   // BN-eval sweeps plain NCHW tensors in place
    const size_t ox = stg ? sg.add(x) : kNoStage;
    const size_t ow = stg && W && W->ndim >= 2 ? sg.add(W) : kNoStage;
    const size_t oy = stg ? sg.add(y) : kNoStage;
    size_t fb = 0;
    if (pl.kind == MS_CONV2D || pl.kind == MS_LINEAR || pl.kind == MS_CONV_TRANSPOSE2D || pl.kind == MS_CONV3D ||
        pl.kind == MS_CONV_TRANSPOSE3D)
        fb = pl.kind == MS_CONV_TRANSPOSE2D    ? ms::conv_dgrad_workspace(pl.dtype, pl.g)
             : pl.kind == MS_CONV3D            ? ms::conv3d_fwd_workspace(pl.dtype, pl.q)
             : pl.kind == MS_CONV_TRANSPOSE3D ? ms::conv3d_dgrad_workspace(pl.dtype, pl.q)
                                               : ms::conv_fwd_workspace(pl.dtype, pl.g);
    char *base = nullptr;
    if (sg.bytes + fb) {
        int werr = 0;
        base = static_cast<char *>(ms::workspace_get(stream, sg.bytes + fb, &werr));
        if (!base) return werr == 1 ? fail(MS_E_NOMEM, "workspace of %zu bytes unavailable", sg.bytes + fb)
                                    : hip_fail(ms::device_last_error(), "workspace");
    }
    void *fws = fb ? base + sg.bytes : nullptr;
    ms_record *r = nullptr;
    if (mask != 0) {
        r = new (std::nothrow) ms_record();
        if (!r) return fail(MS_E_NOMEM, "record allocation failed");
    }
    int err = stage_in(x, base, ox, stream);
    if (!err && ow != kNoStage) err = stage_in(W, base, ow, stream);
    const void *xk = kptr(x, base, ox), *wk = ow != kNoStage ? base + ow : (W ? W->data : nullptr);
    void *yk = kptr(y, base, oy);
    if (!err) switch (pl.kind) {
    case MS_CONV2D:
    case MS_LINEAR:
        err = ms::launch_conv_fwd(pl.dtype, pl.g, xk, wk, b ? b->data : nullptr, yk, fws, stream);
        break;
    case MS_CONV_TRANSPOSE2D:   // the input-gradient contraction of the convolution y -> x, plus b
        err = ms::launch_conv_dgrad(pl.dtype, pl.g, xk, wk, b ? b->data : nullptr, yk, fws, stream);
        break;
    case MS_CONV3D:
        err = ms::launch_conv3d_fwd(pl.dtype, pl.q, x->data, W->data, b ? b->data : nullptr, y->data, fws, stream);
        break;
    case MS_CONV_TRANSPOSE3D:
        err = ms::launch_conv3d_dgrad(pl.dtype, pl.q, x->data, W->data, b ? b->data : nullptr, y->data, fws, stream);
        break;
    case MS_BN_EVAL:
        if (pl.bn_nchw)
            err = ms::launch_bn_nchw(pl.dtype, x->data, layer->running_mean->data, layer->running_var->data,
                                     W ? W->data : nullptr, b ? b->data : nullptr, layer->eps, x->shape[0], pl.C, pl.hw,
                                     y->data, stream, false);
        else
            err = ms::launch_bn_fwd(pl.dtype, xk, layer->running_mean->data, layer->running_var->data,
                                    W ? W->data : nullptr, b ? b->data : nullptr, layer->eps, pl.rows, pl.C, yk, stream);
        break;
    case MS_AVGPOOL:
        err = ms::launch_avgpool_fwd(pl.dtype, xk, pl.Nb, pl.L, pl.C, yk, stream);
        break;
    }
    if (!err) err = stage_out(y, base, oy, stream);
    if (err) {
        delete r;
        return hip_fail(err, "forward launch");
    }
    if (!r) return MS_OK;
    r->magic = kMagic;
    r->plan = pl;
    r->eps = layer->eps;
    r->x = shape_only(x);
    r->y = shape_only(y);
    r->bits = nullptr;
    std::memset(&r->W, 0, sizeof r->W);
    std::memset(&r->b, 0, sizeof r->b);
    std::memset(&r->mean, 0, sizeof r->mean);
    std::memset(&r->var, 0, sizeof r->var);
    if (W) r->W = shape_only(W);
    if (b) r->b = shape_only(b);
    if (pl.kind == MS_BN_EVAL) {
        r->mean = shape_only(layer->running_mean);
        r->var = shape_only(layer->running_var);
    }
    if (borrowed & MS_SAVED_X) r->x.data = x->data;
    if (borrowed & MS_SAVED_W) r->W.data = W->data;
    if (borrowed & MS_SAVED_MEAN) r->mean.data = layer->running_mean->data;
    if (borrowed & MS_SAVED_VAR) r->var.data = layer->running_var->data;
    r->acct = make_account(pl, mask, borrowed, kernels);
    r->consumed = false;
    r->released = false;
    ledger_add(r->acct.saved_activation_bytes);
    g_records.fetch_add(1);
    *rec = r;
    return MS_OK;
}

}  // extern "C"

namespace {

// Backward of a record.  The transient workspace comes from the per-stream
// pool (which may allocate) or, with fixed_scratch, from the library's
// static scratch array (which never does; requests beyond its size fail
// before anything is launched).
ms_status backward_impl(ms_record *r, const ms_tensor *grad_y, const ms_tensor *grad_x,
                        const ms_tensor *grad_W, const ms_tensor *grad_b, void *stream, bool fixed_scratch) {
    clear_err();
    if (!r) return fail(MS_E_NULL, "record is NULL");
    if (r->magic != kMagic) return fail(MS_E_ARG, "not a live record");
    if (r->consumed) return fail(MS_E_CONSUMED, "backward already ran on this record");
    const uint32_t mask = r->acct.mask;
    const Plan &pl = r->plan;
    if ((grad_x != nullptr) != bool(mask & MS_RG_INPUT))
        return fail(MS_E_MASK, "grad_x must be given exactly when the INPUT bit is set");
    if ((grad_W != nullptr) != bool(mask & MS_RG_WEIGHT))
        return fail(MS_E_MASK, "grad_W must be given exactly when the WEIGHT bit is set");
    if ((grad_b != nullptr) != bool(mask & MS_RG_BIAS))
        return fail(MS_E_MASK, "grad_b must be given exactly when the BIAS bit is set");
    ms_status st = check_grad(grad_y, &r->y, "grad_y", pl.kind, false);
    if (st) return st;
    if (grad_x && (st = check_grad(grad_x, &r->x, "grad_x", pl.kind, true))) return st;
    if (grad_W && (st = check_grad(grad_W, &r->W, "grad_W", pl.kind, true))) return st;
    if (grad_b && (st = check_grad(grad_b, &r->b, "grad_b", pl.kind, true))) return st;

    const uint32_t kernels = r->acct.kernels;
    // stand-ins of tensors in other layouts, then the kernels' workspace
    Stager sg;
    // BN-eval wanting dx alone on plain NCHW tensors: the in-place sweep
    const bool bn_native = pl.kind == MS_BN_EVAL && kernels == MS_K_DGRAD && grad_y->ndim == 4 && !canonical(grad_y) &&
                           is_nchw(grad_y) && !canonical(grad_x) && is_nchw(grad_x);
    const bool stg = stageable(pl.kind) && !bn_native;
    const bool x_read = (kernels & MS_K_WGRAD) && pl.kind != MS_AVGPOOL;   // weight gradient (BN: dgamma)
    const bool w_read = (kernels & MS_K_DGRAD) && pl.kind != MS_BN_EVAL && pl.kind != MS_AVGPOOL;
    const size_t ody = stg ? sg.add(grad_y) : kNoStage;
    const size_t ox = stg && x_read ? sg.add(&r->x) : kNoStage;
    const size_t ow = stg && w_read ? sg.add(&r->W) : kNoStage;
    const size_t ogx = stg && grad_x ? sg.add(grad_x) : kNoStage;
    const size_t ogw = stg && grad_W && grad_W->ndim >= 2 ? sg.add(grad_W) : kNoStage;
    const size_t kb = backward_workspace(pl, kernels);
    const size_t ws_bytes = sg.bytes + kb;
    char *base = nullptr;
    if (ws_bytes && fixed_scratch) {
        int werr = 0;
        base = static_cast<char *>(ms::scratch_get(ws_bytes, &werr));
        if (!base) return werr == 1 ? fail(MS_E_UNSUPPORTED, "backward needs %zu bytes of scratch; the fixed scratch "
                                                             "holds %zu", ws_bytes, ms::kScratchBytes)
                                    : hip_fail(ms::device_last_error(), "scratch lookup");
    } else if (ws_bytes) {
        int werr = 0;
        base = static_cast<char *>(ms::workspace_get(stream, ws_bytes, &werr));
        if (!base) return werr == 1 ? fail(MS_E_NOMEM, "workspace of %zu bytes unavailable", ws_bytes)
                                    : hip_fail(ms::device_last_error(), "workspace");
    }
    void *ws = kb ? base + sg.bytes : nullptr;
    int err = stage_in(grad_y, base, ody, stream);
    if (!err) err = stage_in(&r->x, base, ox, stream);
    if (!err) err = stage_in(&r->W, base, ow, stream);
    const void *dy = kptr(grad_y, base, ody);
    const void *xk = ox != kNoStage ? base + ox : r->x.data;
    const void *wk = ow != kNoStage ? base + ow : r->W.data;
    void *gx = kptr(grad_x, base, ogx), *gw = kptr(grad_W, base, ogw);
    if (!err) switch (pl.kind) {
    case MS_CONV2D:
    case MS_LINEAR:
    {
        // the bias gradient rides on the weight gradient when there is one,
        // else (where it can) on the input gradient
        bool db_done = false;
        void *db_dgrad = (kernels & MS_K_BGRAD) && !(kernels & MS_K_WGRAD) ? grad_b->data : nullptr;
        if (!err && (kernels & MS_K_DGRAD))
            err = ms::launch_conv_dgrad(pl.dtype, pl.g, dy, wk, nullptr, gx, ws, stream, db_dgrad, &db_done);
        if (!err && (kernels & MS_K_WGRAD))
            err = ms::launch_conv_wgrad(pl.dtype, pl.g, dy, xk, gw, (kernels & MS_K_BGRAD) ? grad_b->data : nullptr, ws,
                                        stream, &db_done);
        if (!err && (kernels & MS_K_BGRAD) && !db_done)
            err = ms::launch_colsum(pl.dtype, dy, pl.rows, pl.g.K, grad_b->data, ws, stream);
    }
        break;
    case MS_CONV_TRANSPOSE2D:
    {
        // adjoint of the convolution g (input y-shaped, output x-shaped): the
        // input gradient is g's forward of grad_y; the weight gradient is g's
        // weight gradient with x as its output gradient and grad_y as its input
        bool db_unused = false;
        if (kernels & MS_K_DGRAD) err = ms::launch_conv_fwd(pl.dtype, pl.g, dy, wk, nullptr, gx, ws, stream);
        if (!err && (kernels & MS_K_WGRAD))
            err = ms::launch_conv_wgrad(pl.dtype, pl.g, xk, dy, gw, nullptr, ws, stream, &db_unused);
        if (!err && (kernels & MS_K_BGRAD))
            err = ms::launch_colsum(pl.dtype, dy, pl.rows, pl.g.C, grad_b->data, ws, stream);
    }
        break;
    case MS_CONV3D:
    {
        bool db_done = false;
        if (kernels & MS_K_DGRAD)
            err = ms::launch_conv3d_dgrad(pl.dtype, pl.q, dy, r->W.data, nullptr, grad_x->data, ws, stream);
        if (!err && (kernels & MS_K_WGRAD))
            err = ms::launch_conv3d_wgrad(pl.dtype, pl.q, dy, r->x.data, grad_W->data,
                                          (kernels & MS_K_BGRAD) ? grad_b->data : nullptr, ws, stream, &db_done);
        if (!err && (kernels & MS_K_BGRAD) && !db_done)
            err = ms::launch_colsum(pl.dtype, dy, pl.rows, pl.C, grad_b->data, ws, stream);
    }
        break;
    case MS_CONV_TRANSPOSE3D:
    {
        // adjoint of the 3-D convolution q (input y-shaped, output x-shaped)
        bool db_unused = false;
        if (kernels & MS_K_DGRAD)
            err = ms::launch_conv3d_fwd(pl.dtype, pl.q, dy, r->W.data, nullptr, grad_x->data, ws, stream);
        if (!err && (kernels & MS_K_WGRAD))
            err = ms::launch_conv3d_wgrad(pl.dtype, pl.q, r->x.data, dy, grad_W->data, nullptr, ws, stream, &db_unused);
        if (!err && (kernels & MS_K_BGRAD))
            err = ms::launch_colsum(pl.dtype, dy, pl.rows, pl.C, grad_b->data, ws, stream);
    }
        break;
    case MS_BN_EVAL:
        if (bn_native) {
            err = ms::launch_bn_nchw(pl.dtype, dy, nullptr, r->var.data, r->W.data, nullptr, r->eps, r->x.shape[0], pl.C,
                                     pl.hw, gx, stream, true);
            break;
        }
        err = ms::launch_bn_bwd(pl.dtype, dy, (kernels & MS_K_WGRAD) ? xk : nullptr,
                                (kernels & MS_K_WGRAD) ? r->mean.data : nullptr, r->var.data,
                                (kernels & MS_K_DGRAD) ? r->W.data : nullptr, r->eps, pl.rows, pl.C,
                                gx, grad_W ? grad_W->data : nullptr, grad_b ? grad_b->data : nullptr, ws, stream);
        break;
    case MS_AVGPOOL:
        if (kernels & MS_K_DGRAD) err = ms::launch_avgpool_bwd(pl.dtype, dy, pl.Nb, pl.L, pl.C, gx, stream);
        break;
    case MS_RELU:
        if (kernels & MS_K_DGRAD) err = ms::launch_relu_bwd(pl.dtype, dy, r->bits, pl.n, grad_x->data, stream);
        break;
    case MS_DROPOUT:   // the mask is drawn again from the record's key and counter
        if (kernels & MS_K_DGRAD)
            err = ms::launch_dropout(pl.dtype, dy, pl.n, grad_x->data, r->seed, r->offset, r->thresh, r->scale,
                                     r->drop_all, stream);
        break;
    }
    if (!err) err = stage_out(grad_x, base, ogx, stream);
    if (!err) err = stage_out(grad_W, base, ogw, stream);
    if (err) return hip_fail(err, "backward launch");
    r->consumed = true;
    release(r);
    return MS_OK;
}

// Profiling events stay off for the calling thread while one lives.
struct ProfOff {
    ProfOff() { ms::prof_thread_off(true); }
    ~ProfOff() { ms::prof_thread_off(false); }
};

}  // namespace

extern "C" {

ms_status ms_layer_backward(ms_record *r, const ms_tensor *grad_y, const ms_tensor *grad_x,
                            const ms_tensor *grad_W, const ms_tensor *grad_b, void *stream) {
    return backward_impl(r, grad_y, grad_x, grad_W, grad_b, stream, false);
}

ms_status ms_layer_backward_noalloc(ms_record *r, const ms_tensor *grad_y, const ms_tensor *grad_x,
                                    const ms_tensor *grad_W, const ms_tensor *grad_b, void *stream) {
    ProfOff off;
    return backward_impl(r, grad_y, grad_x, grad_W, grad_b, stream, true);
}

uint64_t ms_noalloc_scratch_bytes(void) { return ms::kScratchBytes; }

uint64_t ms_relu_mask_bytes(int64_t n) { return relu_mask_bytes(n); }

ms_status ms_relu_forward(const ms_tensor *x, const ms_tensor *y, void *bits, uint32_t mask, ms_record **rec,
                          void *stream) {
    clear_err();
    if (!rec) return fail(MS_E_NULL, "rec is NULL");
    *rec = nullptr;
    if (!y) return fail(MS_E_NULL, "y is NULL");
    ms_layer layer{};
    layer.kind = MS_RELU;
    Plan pl;
    ms_status st = validate_forward(&layer, x, nullptr, nullptr, mask, y, true, &pl);
    if (st) return st;
    const bool keep = mask & MS_RG_INPUT;
    if (keep && pl.bits_bytes > 0 && !bits) return fail(MS_E_NULL, "bits is NULL but the INPUT bit is set");
    if (keep && (reinterpret_cast<uintptr_t>(bits) & 3u)) return fail(MS_E_ARG, "bits must be 4-byte aligned");
    ms_record *r = nullptr;
    if (keep) {
        r = new (std::nothrow) ms_record();
        if (!r) return fail(MS_E_NOMEM, "record allocation failed");
    }
    // without a record the mask is not needed: the forward writes y only
    const int err = pl.n == 0 && !keep ? 0
                    : ms::launch_relu_fwd(pl.dtype, x->data, pl.n, y->data, keep ? bits : nullptr,
                                          keep ? (int64_t)pl.bits_bytes : 0, stream);
    if (err) {
        delete r;
        return hip_fail(err, "forward launch");
    }
    if (!r) return MS_OK;
    const uint32_t borrowed = borrowed_bits(MS_RELU, mask, MS_POLICY_SELECTIVE, false, false);
    const uint32_t kernels = kernel_bits(MS_RELU, mask);
    r->magic = kMagic;
    r->plan = pl;
    r->eps = 0.f;
    r->x = shape_only(x);
    r->y = shape_only(y);
    std::memset(&r->W, 0, sizeof r->W);
    std::memset(&r->b, 0, sizeof r->b);
    std::memset(&r->mean, 0, sizeof r->mean);
    std::memset(&r->var, 0, sizeof r->var);
    r->bits = bits;
    r->acct = make_account(pl, mask, borrowed, kernels);
    r->consumed = false;
    r->released = false;
    ledger_add(r->acct.saved_activation_bytes);
    g_records.fetch_add(1);
    *rec = r;
    return MS_OK;
}

uint64_t ms_dropout_blocks(int64_t n) { return n > 0 ? (uint64_t)((n + 3) / 4) : 0u; }

ms_status ms_dropout_forward(const ms_tensor *x, const ms_tensor *y, float p, uint64_t seed, uint64_t offset,
                             uint32_t mask, ms_record **rec, void *stream) {
    clear_err();
    if (!rec) return fail(MS_E_NULL, "rec is NULL");
    *rec = nullptr;
    if (!y) return fail(MS_E_NULL, "y is NULL");
    if (!(p >= 0.f && p <= 1.f)) return fail(MS_E_ARG, "p must be finite and in [0, 1]");
    ms_layer layer{};
    layer.kind = MS_DROPOUT;
    Plan pl;
    ms_status st = validate_forward(&layer, x, nullptr, nullptr, mask, y, true, &pl);
    if (st) return st;
    // keep iff the element's word >= floor(p * 2^32); p < 1 keeps that below 2^32
    const int drop_all = p == 1.f;
    const uint32_t thresh = drop_all ? 0u : (uint32_t)std::floor((double)p * 4294967296.0);
    const float scale = drop_all ? 0.f : (float)(1.0 / (1.0 - (double)p));
    const bool keep = mask & MS_RG_INPUT;
    ms_record *r = nullptr;
    if (keep) {
        r = new (std::nothrow) ms_record();
        if (!r) return fail(MS_E_NOMEM, "record allocation failed");
    }
    const int err = ms::launch_dropout(pl.dtype, x->data, pl.n, y->data, seed, offset, thresh, scale, drop_all, stream);
    if (err) {
        delete r;
        return hip_fail(err, "forward launch");
    }
    if (!r) return MS_OK;
    r->magic = kMagic;
    r->plan = pl;
    r->eps = 0.f;
    r->x = shape_only(x);
    r->y = shape_only(y);
    std::memset(&r->W, 0, sizeof r->W);
    std::memset(&r->b, 0, sizeof r->b);
    std::memset(&r->mean, 0, sizeof r->mean);
    std::memset(&r->var, 0, sizeof r->var);
    r->bits = nullptr;
    r->seed = seed;
    r->offset = offset;
    r->thresh = thresh;
    r->scale = scale;
    r->drop_all = drop_all;
    r->acct = make_account(pl, mask, borrowed_bits(MS_DROPOUT, mask, MS_POLICY_SELECTIVE, false, false),
                           kernel_bits(MS_DROPOUT, mask));
    r->consumed = false;
    r->released = false;
    ledger_add(r->acct.saved_activation_bytes);
    g_records.fetch_add(1);
    *rec = r;
    return MS_OK;
}

ms_status ms_record_account(const ms_record *r, ms_account *out) {
    clear_err();
    if (!r || !out) return fail(MS_E_NULL, "NULL argument");
    if (r->magic != kMagic) return fail(MS_E_ARG, "not a live record");
    *out = r->acct;
    return MS_OK;
}

void ms_record_free(ms_record *r) {
    if (!r || r->magic != kMagic) return;
    release(r);
    r->magic = 0;
    g_records.fetch_sub(1);
    delete r;
}

ms_status ms_ledger_read(uint64_t *live, uint64_t *peak) {
    clear_err();
    if (!live || !peak) return fail(MS_E_NULL, "NULL argument");
    *live = g_live.load();
    *peak = g_peak.load();
    return MS_OK;
}

ms_status ms_ledger_reset(void) {
    clear_err();
    g_peak.store(g_live.load());
    return MS_OK;
}

ms_status ms_policy_account(const ms_layer *layer, const ms_tensor *x, const ms_tensor *W,
                            const ms_tensor *b, uint32_t mask, int32_t policy, ms_account *out) {
    clear_err();
    if (!out) return fail(MS_E_NULL, "out is NULL");
    if (policy < MS_POLICY_SELECTIVE || policy > MS_POLICY_ALL_TRUE) return fail(MS_E_ARG, "unknown policy");
    Plan pl;
    ms_status st = validate_forward(layer, x, W, b, mask, nullptr, false, &pl);
    if (st) return st;
    uint32_t eff = mask;
    if (policy == MS_POLICY_ALL_TRUE) {
        eff = MS_RG_INPUT;
        if (pl.kind != MS_AVGPOOL) eff |= (W ? (uint32_t)MS_RG_WEIGHT : 0u) | (b ? (uint32_t)MS_RG_BIAS : 0u);
    }
    const uint32_t borrowed = borrowed_bits(pl.kind, mask, policy, pl.has_w, pl.has_b);
    *out = make_account(pl, eff, borrowed, kernel_bits(pl.kind, eff));
    return MS_OK;
}

ms_status ms_profile_start(uint32_t kinds) {
    clear_err();
    if (kinds & ~63u) return fail(MS_E_ARG, "unknown profile kinds 0x%x", kinds);
    const int err = ms::prof_start(kinds);
    return err ? hip_fail(err, "ms_profile_start") : MS_OK;
}

ms_status ms_profile_read(uint32_t kind, uint64_t *launches, double *total_ms) {
    clear_err();
    if (!launches || !total_ms) return fail(MS_E_NULL, "NULL argument");
    if (kind != MS_PROF_FWD && kind != MS_PROF_DGRAD && kind != MS_PROF_WGRAD && kind != MS_PROF_BN &&
        kind != MS_PROF_ACT && kind != MS_PROF_RED)
        return fail(MS_E_ARG, "read one kind at a time");
    const int err = ms::prof_read(kind, launches, total_ms);
    return err ? hip_fail(err, "ms_profile_read") : MS_OK;
}

const char *ms_status_str(int32_t s) {
    switch (s) {
    case MS_OK: return "ok";
    case MS_E_NULL: return "null pointer";
    case MS_E_MASK: return "invalid mask or gradient set";
    case MS_E_SHAPE: return "shape mismatch";
    case MS_E_DTYPE: return "unsupported dtype";
    case MS_E_LAYOUT: return "unsupported memory layout";
    case MS_E_UNSUPPORTED: return "unsupported configuration";
    case MS_E_CONSUMED: return "record already consumed";
    case MS_E_NOMEM: return "out of device memory";
    case MS_E_HIP: return "HIP error";
    case MS_E_ARG: return "invalid argument";
    default: return "unknown status";
    }
}

const char *ms_last_error(void) { return g_err.c_str(); }

const char *ms_version(void) { return "memsave-gfx950 0.1.0"; }

void ms_testing_fail_next_workspace(int32_t n) { ms::workspace_fail_next(n); }

int64_t ms_testing_live_records(void) { return g_records.load(); }

int32_t ms_testing_gemm_plan(int32_t pass, const int32_t geom[13], int32_t out[10]) {
    if (!geom || !out) return -1;
    const ms::ConvGeom g{geom[0], geom[1], geom[2], geom[3], geom[4], geom[5], geom[6],
                         geom[7], geom[8], geom[9], geom[10], geom[11], geom[12]};
    int o[10];
    const int r = ms::gemm_plan_info(pass, g, o);
    for (int i = 0; i < 10; ++i) out[i] = o[i];
    return r;
}

}  // extern "C"

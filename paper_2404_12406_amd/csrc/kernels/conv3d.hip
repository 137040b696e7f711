// 3-D convolution and its transpose by folding the depth axis into the
// 2-D implicit GEMMs (App. B of the paper probes torch.nn.Conv3d and
// ConvTranspose3d; Sec. 2.2.1's rule applies to them as to Conv2d).
//
// A 3-D convolution u[N][Din][H][W][C] -> v[N][Do][P][Q][K] with filter
// W[K][T][R][S][C] (depth taps T, stride sd, pad pd) is the 2-D convolution
// over N*Do images of
//     fold(u)[(n, o)][h][w][t*C + c] = u[n][o*sd - pd + t][h][w][c]   (0 outside [0, Din))
// with the filter's taps regrouped as Wc[K][R][S][T*C].  So:
//   forward          v  = conv2d(fold(u), Wc)
//   input gradient   du = unfold_sum(conv2d_input_grad(dv, Wc)),
//                    unfold_sum(U)[n][d][h][w][c] = sum over (t, o) with
//                    o*sd - pd + t = d of U[(n, o)][h][w][t*C + c]
//   weight gradient  dW = regroup^-1(conv2d_weight_grad(dv, fold(u)))
// The transposed 3-D convolution is the adjoint of such a convolution: its
// forward is the input-gradient path (plus its bias, added by unfold_sum),
// its input gradient the forward path, its weight gradient the weight-
// gradient path with its input in the role of dv.
//
// The fold buffer is T / sd times the input; it lives in transient
// workspace for one call.  The three kernels here are streaming passes.
#include <algorithm>

#include "common.h"
#include "../device.h"

namespace ms {
namespace {

size_t al256(size_t n) { return (n + 255) / 256 * 256; }

int blocks_for(int64_t work) {
    return (int)std::max<int64_t>(1, std::min<int64_t>((work + 255) / 256, 65536));
}

// V consecutive channels: one 16-byte vector when V * sizeof(T) == 16.
template <typename T, int V>
struct Chan {
    T e[V];
    __device__ __forceinline__ void load(const T *p) {
        if constexpr (V * sizeof(T) == 16) *reinterpret_cast<u32x4 *>(e) = *reinterpret_cast<const u32x4 *>(p);
        else
#pragma unroll
            for (int k = 0; k < V; ++k) e[k] = p[k];
    }
    __device__ __forceinline__ void store(T *p) const {
        if constexpr (V * sizeof(T) == 16) *reinterpret_cast<u32x4 *>(p) = *reinterpret_cast<const u32x4 *>(e);
        else
#pragma unroll
            for (int k = 0; k < V; ++k) p[k] = e[k];
    }
};

// fold: out[(n*Do + o)*HW + hw][t*C + c] = in[(n*Din + o*sd - pd + t)*HW + hw][c] or 0.
// A thread moves V channels (16 bytes when C is a multiple of V) of one
// (output pixel, tap); indices are 32-bit (every buffer has fewer than 2^31
// elements).
template <typename T, int V>
__global__ __launch_bounds__(256) void depth_fold_kernel(const T *__restrict__ in, T *__restrict__ out, int N,
                                                         int Din, int Do, int HW, int C, int Tt, int sd, int pd) {
    const uint32_t cv = (uint32_t)(C / V);                  // vectors per channel run
    const uint32_t per_pix = (uint32_t)Tt * cv;             // vectors per folded pixel row
    const uint32_t total = (uint32_t)N * Do * HW * per_pix;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const uint32_t pix = i / per_pix, j = i - pix * per_pix;   // pix = (n*Do + o)*HW + hw
        const uint32_t t = j / cv, c0 = (j - t * cv) * V;
        const uint32_t img = pix / (uint32_t)HW, hw = pix - img * (uint32_t)HW;
        const uint32_t n = img / (uint32_t)Do, o = img - n * (uint32_t)Do;
        const int d = (int)o * sd - pd + (int)t;
        Chan<T, V> v;
        if (d >= 0 && d < Din) {
            v.load(in + ((size_t)(n * (uint32_t)Din + (uint32_t)d) * HW + hw) * C + c0);
        } else {
#pragma unroll
            for (int k = 0; k < V; ++k) v.e[k] = (T)0.f;
        }
        v.store(out + (size_t)pix * (Tt * C) + t * C + c0);
    }
}

// unfold_sum: out[(n*Dout + d)*HW + hw][c] = bias[c] + sum over t with
// o = (d + pd - t) / sd an integer in [0, Dc) of in[(n*Dc + o)*HW + hw][t*C + c],
// summed in fp32 and rounded once.  A thread owns V channels of one output
// pixel.
template <typename T, int V>
__global__ __launch_bounds__(256) void depth_unfold_sum_kernel(const T *__restrict__ in, T *__restrict__ out,
                                                               const T *__restrict__ bias, int N, int Dc, int Dout,
                                                               int HW, int C, int Tt, int sd, int pd) {
    const uint32_t cv = (uint32_t)(C / V);
    const uint32_t total = (uint32_t)N * Dout * HW * cv;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const uint32_t pix = i / cv, c0 = (i - pix * cv) * V;      // pix = (n*Dout + d)*HW + hw
        const uint32_t img = pix / (uint32_t)HW, hw = pix - img * (uint32_t)HW;
        const uint32_t n = img / (uint32_t)Dout, d = img - n * (uint32_t)Dout;
        float acc[V];
#pragma unroll
        for (int k = 0; k < V; ++k) acc[k] = bias ? to_f32(bias[c0 + k]) : 0.f;
        for (int t = 0; t < Tt; ++t) {
            const int q = (int)d + pd - t;
            if (q < 0 || q % sd != 0) continue;
            const int o = q / sd;
            if (o >= Dc) continue;
            Chan<T, V> v;
            v.load(in + ((size_t)(n * (uint32_t)Dc + (uint32_t)o) * HW + hw) * (Tt * C) + t * C + c0);
#pragma unroll
            for (int k = 0; k < V; ++k) acc[k] += to_f32(v.e[k]);
        }
        Chan<T, V> r;
#pragma unroll
        for (int k = 0; k < V; ++k) r.e[k] = from_f32<T>(acc[k]);
        r.store(out + (size_t)pix * C + c0);
    }
}

// Tap regrouping of a filter with K rows: [K][T][RS][C] <-> [K][RS][T][C].
template <typename T>
__global__ __launch_bounds__(256) void regroup_taps_kernel(const T *__restrict__ src, T *__restrict__ dst, int64_t K,
                                                           int64_t Tt, int64_t RS, int64_t C, int to_folded) {
    const int64_t total = K * Tt * RS * C;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        int64_t r = i;
        const int64_t c = r % C;
        r /= C;
        const int64_t rs = r % RS;
        r /= RS;
        const int64_t t = r % Tt;
        const int64_t k = r / Tt;
        const int64_t a = ((k * Tt + t) * RS + rs) * C + c;   // [K][T][RS][C]
        const int64_t b = ((k * RS + rs) * Tt + t) * C + c;   // [K][RS][T][C]
        if (to_folded) dst[b] = src[a];
        else dst[a] = src[b];
    }
}

bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <typename T>
int fold_t(const Conv3dGeom &q, const void *u, void *out, hipStream_t st) {
    const int HW = q.g.H * q.g.W;
    constexpr int V = 16 / sizeof(T);
    const bool vec = q.C % V == 0 && al16(u) && al16(out);
    const int64_t work = (int64_t)q.N * q.Do * HW * q.T * (vec ? q.C / V : q.C);
    if (work == 0) return 0;
    if (vec)
        hipLaunchKernelGGL((depth_fold_kernel<T, V>), dim3(blocks_for(work)), dim3(256), 0, st, (const T *)u, (T *)out,
                           q.N, q.Din, q.Do, HW, q.C, q.T, q.sd, q.pd);
    else
        hipLaunchKernelGGL((depth_fold_kernel<T, 1>), dim3(blocks_for(work)), dim3(256), 0, st, (const T *)u, (T *)out,
                           q.N, q.Din, q.Do, HW, q.C, q.T, q.sd, q.pd);
    return (int)hipGetLastError();
}

template <typename T>
int unfold_t(const Conv3dGeom &q, const void *in, const void *bias, void *out, hipStream_t st) {
    const int HW = q.g.H * q.g.W;
    constexpr int V = 16 / sizeof(T);
    const bool vec = q.C % V == 0 && al16(in) && al16(out);
    const int64_t work = (int64_t)q.N * q.Din * HW * (vec ? q.C / V : q.C);
    if (work == 0) return 0;
    if (vec)
        hipLaunchKernelGGL((depth_unfold_sum_kernel<T, V>), dim3(blocks_for(work)), dim3(256), 0, st, (const T *)in,
                           (T *)out, (const T *)bias, q.N, q.Do, q.Din, HW, q.C, q.T, q.sd, q.pd);
    else
        hipLaunchKernelGGL((depth_unfold_sum_kernel<T, 1>), dim3(blocks_for(work)), dim3(256), 0, st, (const T *)in,
                           (T *)out, (const T *)bias, q.N, q.Do, q.Din, HW, q.C, q.T, q.sd, q.pd);
    return (int)hipGetLastError();
}

template <typename T>
int regroup_t(const Conv3dGeom &q, const void *src, void *dst, int to_folded, hipStream_t st) {
    const int64_t RS = (int64_t)q.g.R * q.g.S;
    const int64_t work = (int64_t)q.g.K * q.T * RS * q.C;
    if (work == 0) return 0;
    hipLaunchKernelGGL((regroup_taps_kernel<T>), dim3(blocks_for(work)), dim3(256), 0, st, (const T *)src, (T *)dst,
                       (int64_t)q.g.K, (int64_t)q.T, RS, (int64_t)q.C, to_folded);
    return (int)hipGetLastError();
}

int fold(int dtype, const Conv3dGeom &q, const void *u, void *out, hipStream_t st) {
    return dtype == kBF16 ? fold_t<bf16>(q, u, out, st) : fold_t<float>(q, u, out, st);
}
int unfold(int dtype, const Conv3dGeom &q, const void *in, const void *bias, void *out, hipStream_t st) {
    return dtype == kBF16 ? unfold_t<bf16>(q, in, bias, out, st) : unfold_t<float>(q, in, bias, out, st);
}
int regroup(int dtype, const Conv3dGeom &q, const void *src, void *dst, int to_folded, hipStream_t st) {
    return dtype == kBF16 ? regroup_t<bf16>(q, src, dst, to_folded, st) : regroup_t<float>(q, src, dst, to_folded, st);
}

size_t elt(int dtype) { return dtype == kBF16 ? 2 : 4; }
// the folded input [N*Do][H][W][T*C] and the regrouped filter [K][R][S][T*C]
size_t fold_bytes(int dtype, const Conv3dGeom &q) {
    return al256((size_t)q.g.N * q.g.H * q.g.W * q.g.C * elt(dtype));
}
size_t filter_bytes(int dtype, const Conv3dGeom &q) {
    return al256((size_t)q.g.K * q.g.R * q.g.S * q.g.C * elt(dtype));
}

}  // namespace

size_t conv3d_fwd_workspace(int dtype, const Conv3dGeom &q) {
    return fold_bytes(dtype, q) + filter_bytes(dtype, q) + al256(conv_fwd_workspace(dtype, q.g));
}

size_t conv3d_dgrad_workspace(int dtype, const Conv3dGeom &q) {
    return fold_bytes(dtype, q) + filter_bytes(dtype, q) + al256(conv_dgrad_workspace(dtype, q.g));
}

size_t conv3d_wgrad_workspace(int dtype, const Conv3dGeom &q, bool with_db) {
    return fold_bytes(dtype, q) + filter_bytes(dtype, q) + al256(conv_wgrad_workspace(dtype, q.g, with_db));
}

int launch_conv3d_fwd(int dtype, const Conv3dGeom &q, const void *u, const void *w, const void *bias, void *v,
                      void *ws, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    char *p = static_cast<char *>(ws);
    void *uf = p, *wc = p + fold_bytes(dtype, q), *rest = p + fold_bytes(dtype, q) + filter_bytes(dtype, q);
    int err = fold(dtype, q, u, uf, st);
    if (!err) err = regroup(dtype, q, w, wc, 1, st);
    if (!err) err = launch_conv_fwd(dtype, q.g, uf, wc, bias, v, rest, stream);
    return err;
}

int launch_conv3d_dgrad(int dtype, const Conv3dGeom &q, const void *dv, const void *w, const void *bias, void *du,
                        void *ws, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    char *p = static_cast<char *>(ws);
    void *uf = p, *wc = p + fold_bytes(dtype, q), *rest = p + fold_bytes(dtype, q) + filter_bytes(dtype, q);
    int err = regroup(dtype, q, w, wc, 1, st);
    if (!err) err = launch_conv_dgrad(dtype, q.g, dv, wc, nullptr, uf, rest, stream);
    if (!err) err = unfold(dtype, q, uf, bias, du, st);
    return err;
}

int launch_conv3d_wgrad(int dtype, const Conv3dGeom &q, const void *dv, const void *u, void *dw, void *db, void *ws,
                        void *stream, bool *db_done) {
    hipStream_t st = (hipStream_t)stream;
    char *p = static_cast<char *>(ws);
    void *uf = p, *wc = p + fold_bytes(dtype, q), *rest = p + fold_bytes(dtype, q) + filter_bytes(dtype, q);
    int err = fold(dtype, q, u, uf, st);
    if (!err) err = launch_conv_wgrad(dtype, q.g, dv, uf, wc, db, rest, stream, db_done);
    if (!err) err = regroup(dtype, q, wc, dw, 0, st);
    return err;
}

}  // namespace ms

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

// fold: out[(n*Do + o)*HW + hw][t*C + c] = in[(n*Din + o*sd - pd + t)*HW + hw][c] or 0.
// V elements per thread step (16 bytes when C is a multiple of V).
template <typename T, int V>
__global__ __launch_bounds__(256) void depth_fold_kernel(const T *__restrict__ in, T *__restrict__ out, int64_t N,
                                                         int64_t Din, int64_t Do, int64_t HW, int64_t C, int64_t Tt,
                                                         int64_t sd, int64_t pd) {
    const int64_t cv = C / V;                      // vectors per channel run
    const int64_t total = N * Do * HW * Tt * cv;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        int64_t r = i;
        const int64_t c0 = (r % cv) * V;
        r /= cv;
        const int64_t t = r % Tt;
        r /= Tt;
        const int64_t hw = r % HW;
        r /= HW;
        const int64_t o = r % Do;
        const int64_t n = r / Do;
        const int64_t d = o * sd - pd + t;
        T *dst = out + ((n * Do + o) * HW + hw) * (Tt * C) + t * C + c0;
        if (d >= 0 && d < Din) {
            const T *src = in + ((n * Din + d) * HW + hw) * C + c0;
            if constexpr (V * sizeof(T) == 16) {
                *reinterpret_cast<u32x4 *>(dst) = *reinterpret_cast<const u32x4 *>(src);
            } else {
#pragma unroll
                for (int e = 0; e < V; ++e) dst[e] = src[e];
            }
        } else {
            if constexpr (V * sizeof(T) == 16) {
                *reinterpret_cast<u32x4 *>(dst) = u32x4{0u, 0u, 0u, 0u};
            } else {
#pragma unroll
                for (int e = 0; e < V; ++e) dst[e] = (T)0.f;
            }
        }
    }
}

// unfold_sum: out[(n*Dout + d)*HW + hw][c] = bias[c] + sum over t with
// o = (d + pd - t) / sd an integer in [0, Dc) of in[(n*Dc + o)*HW + hw][t*C + c],
// summed in fp32 and rounded once.
template <typename T>
__global__ __launch_bounds__(256) void depth_unfold_sum_kernel(const T *__restrict__ in, T *__restrict__ out,
                                                               const T *__restrict__ bias, int64_t N, int64_t Dc,
                                                               int64_t Dout, int64_t HW, int64_t C, int64_t Tt,
                                                               int64_t sd, int64_t pd) {
    const int64_t total = N * Dout * HW * C;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        int64_t r = i;
        const int64_t c = r % C;
        r /= C;
        const int64_t hw = r % HW;
        r /= HW;
        const int64_t d = r % Dout;
        const int64_t n = r / Dout;
        float acc = bias ? to_f32(bias[c]) : 0.f;
        for (int64_t t = 0; t < Tt; ++t) {
            const int64_t q = d + pd - t;
            if (q < 0 || q % sd != 0) continue;
            const int64_t o = q / sd;
            if (o >= Dc) continue;
            acc += to_f32(in[((n * Dc + o) * HW + hw) * (Tt * C) + t * C + c]);
        }
        out[i] = from_f32<T>(acc);
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

template <typename T>
int fold_t(const Conv3dGeom &q, const void *u, void *out, hipStream_t st) {
    const int64_t HW = (int64_t)q.g.H * q.g.W;
    constexpr int V = 16 / sizeof(T);
    const bool vec = q.C % V == 0 && (reinterpret_cast<uintptr_t>(u) & 15u) == 0 &&
                     (reinterpret_cast<uintptr_t>(out) & 15u) == 0;
    const int64_t work = (int64_t)q.N * q.Do * HW * q.T * (vec ? q.C / V : q.C);
    if (work == 0) return 0;
    if (vec)
        hipLaunchKernelGGL((depth_fold_kernel<T, V>), dim3(blocks_for(work)), dim3(256), 0, st, (const T *)u, (T *)out,
                           (int64_t)q.N, (int64_t)q.Din, (int64_t)q.Do, HW, (int64_t)q.C, (int64_t)q.T, (int64_t)q.sd,
                           (int64_t)q.pd);
    else
        hipLaunchKernelGGL((depth_fold_kernel<T, 1>), dim3(blocks_for(work)), dim3(256), 0, st, (const T *)u, (T *)out,
                           (int64_t)q.N, (int64_t)q.Din, (int64_t)q.Do, HW, (int64_t)q.C, (int64_t)q.T, (int64_t)q.sd,
                           (int64_t)q.pd);
    return (int)hipGetLastError();
}

template <typename T>
int unfold_t(const Conv3dGeom &q, const void *in, const void *bias, void *out, hipStream_t st) {
    const int64_t HW = (int64_t)q.g.H * q.g.W;
    const int64_t work = (int64_t)q.N * q.Din * HW * q.C;
    if (work == 0) return 0;
    hipLaunchKernelGGL((depth_unfold_sum_kernel<T>), dim3(blocks_for(work)), dim3(256), 0, st, (const T *)in, (T *)out,
                       (const T *)bias, (int64_t)q.N, (int64_t)q.Do, (int64_t)q.Din, HW, (int64_t)q.C, (int64_t)q.T,
                       (int64_t)q.sd, (int64_t)q.pd);
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

// ReLU whose backward needs one bit per element (Sec. 2.2.2 of the paper):
// an activation that stores its output keeps the next layer's input alive
// whatever that layer's differentiability mask says, so this ReLU keeps only
// the sign information its input gradient needs.  The paper's version keeps
// a one-byte boolean and names one-bit booleans as the next step; here the
// mask is packed 8 elements per byte, little-endian (bit e of byte j is
// element 8j + e in memory order; the 4 bytes of word w are bytes 4w..4w+3).
//
//   forward:  y = x < 0 ? 0 : x   (NaN and -0 pass through unchanged)
//             bit i = !(y_i <= 0)  (positive or NaN: a NaN passes its
//                                  gradient, as PyTorch's ReLU backward does)
//   backward: dx_i = bit i ? dy_i : 0
//
// Both are one streaming pass: a thread owns groups of 8 consecutive
// elements (one 16-byte vector of bf16, two of fp32) and their mask byte, and
// keeps kU groups' loads in flight.  HBM bytes per element: 2 * elt + 1/8.
#include <algorithm>

#include "common.h"
#include "../device.h"

namespace ms {
namespace {

constexpr int kU = 4;   // groups per thread per pass

// ngroups = ceil(n / 8) mask bytes carry bits; the bytes after them up to
// nbytes (the word-rounded mask size) are written as zeros.  bits == nullptr
// (nbytes == 0): y only.
template <typename T, bool VEC>
__global__ __launch_bounds__(256) void relu_fwd_kernel(const T *__restrict__ x, T *__restrict__ y,
                                                       uint8_t *__restrict__ bits, int64_t n, int64_t ngroups,
                                                       int64_t nbytes) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t v0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; v0 < ngroups; v0 += kU * stride) {
        Group8<T> g[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u)
            if (v0 + u * stride < ngroups) g[u] = load_group8<T, VEC>(x, (v0 + u * stride) * 8, n);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int64_t v = v0 + u * stride;
            if (v >= ngroups) continue;
            uint32_t byte = 0;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float f = to_f32(g[u].e[e]);
                if (f < 0.f) g[u].e[e] = (T)0.f;
                byte |= (f <= 0.f ? 0u : 1u) << e;
            }
            store_group8<T, VEC>(y, v * 8, n, g[u]);
            if (bits) bits[v] = (uint8_t)byte;   // no mask without a record
        }
    }
    if (blockIdx.x == 0 && threadIdx.x < nbytes - ngroups) bits[ngroups + threadIdx.x] = 0;
}

template <typename T, bool VEC>
__global__ __launch_bounds__(256) void relu_bwd_kernel(const T *__restrict__ dy, const uint8_t *__restrict__ bits,
                                                       T *__restrict__ dx, int64_t n, int64_t ngroups) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t v0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; v0 < ngroups; v0 += kU * stride) {
        Group8<T> g[kU];
        uint32_t byte[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int64_t v = v0 + u * stride;
            byte[u] = 0;
            if (v < ngroups) {
                g[u] = load_group8<T, VEC>(dy, v * 8, n);
                byte[u] = bits[v];
            }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int64_t v = v0 + u * stride;
            if (v >= ngroups) continue;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (!((byte[u] >> e) & 1u)) g[u].e[e] = (T)0.f;
            store_group8<T, VEC>(dx, v * 8, n, g[u]);
        }
    }
}

bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int grid_for(int64_t ngroups) {
    return (int)std::max<int64_t>(1, std::min<int64_t>((ngroups + 256 * kU - 1) / (256 * kU), 65536));
}

template <typename T>
int fwd_t(const void *x, int64_t n, void *y, void *bits, int64_t nbytes, hipStream_t st) {
    const int64_t ng = (n + 7) / 8;
    const bool vec = al16(x) && al16(y);
    if (vec)
        hipLaunchKernelGGL((relu_fwd_kernel<T, true>), dim3(grid_for(ng)), dim3(256), 0, st, (const T *)x, (T *)y,
                           (uint8_t *)bits, n, ng, nbytes);
    else
        hipLaunchKernelGGL((relu_fwd_kernel<T, false>), dim3(grid_for(ng)), dim3(256), 0, st, (const T *)x, (T *)y,
                           (uint8_t *)bits, n, ng, nbytes);
    return (int)hipGetLastError();
}

template <typename T>
int bwd_t(const void *dy, const void *bits, int64_t n, void *dx, hipStream_t st) {
    const int64_t ng = (n + 7) / 8;
    const bool vec = al16(dy) && al16(dx);
    if (vec)
        hipLaunchKernelGGL((relu_bwd_kernel<T, true>), dim3(grid_for(ng)), dim3(256), 0, st, (const T *)dy,
                           (const uint8_t *)bits, (T *)dx, n, ng);
    else
        hipLaunchKernelGGL((relu_bwd_kernel<T, false>), dim3(grid_for(ng)), dim3(256), 0, st, (const T *)dy,
                           (const uint8_t *)bits, (T *)dx, n, ng);
    return (int)hipGetLastError();
}

}  // namespace

int launch_relu_fwd(int dtype, const void *x, int64_t n, void *y, void *bits, int64_t bits_bytes, void *stream) {
    if (n == 0 && bits_bytes == 0) return 0;
    hipStream_t st = (hipStream_t)stream;
    prof_mark(kProfAct, st, true);
    const int err = dtype == kBF16 ? fwd_t<bf16>(x, n, y, bits, bits_bytes, st) : fwd_t<float>(x, n, y, bits, bits_bytes, st);
    prof_mark(kProfAct, st, false);
    return err;
}

int launch_relu_bwd(int dtype, const void *dy, const void *bits, int64_t n, void *dx, void *stream) {
    if (n == 0) return 0;
    hipStream_t st = (hipStream_t)stream;
    prof_mark(kProfAct, st, true);
    const int err = dtype == kBF16 ? bwd_t<bf16>(dy, bits, n, dx, st) : bwd_t<float>(dy, bits, n, dx, st);
    prof_mark(kProfAct, st, false);
    return err;
}

}  // namespace ms

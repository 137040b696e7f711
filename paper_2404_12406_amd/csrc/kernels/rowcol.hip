// Bandwidth-bound kernels over an NHWC activation viewed as [rows][C]
// (rows = N*H*W pixels, C channels contiguous):
//   - BN in evaluation mode, forward y = gamma (x - mu)/sqrt(var + eps) + beta
//     folded per channel into y = x*s + t (s = gamma/sqrt(var+eps),
//     t = beta - mu*s, computed in fp32 by each thread for its channels);
//   - BN-eval backward: dx = dy*s (needs gamma and var, not x),
//     dgamma = sum dy*(x - mu)/sqrt(var+eps) (the only use of x),
//     dbeta = sum dy;
//   - bias gradient of conv / linear: column sums of dy;
//   - global average pool and its adjoint.
//
// Thread map of the reductions: a block is RG x TC threads; thread (rg, tc)
// owns the channel vector tc of its block's column tile for the whole kernel
// and walks rows rg, rg+RG, ... of its block's row chunk, so per-channel
// constants live in registers and a wave reads whole contiguous rows
// (coalesced 16-byte loads).  The BN-eval forward is a linear sweep (below).
// Reductions: per-thread fp32 partials -> LDS reduction over RG -> one fp32
// partial per (row chunk, channel) -> finalize kernel (deterministic order).
#include <algorithm>

#include "common.h"
#include "../device.h"

namespace ms {

namespace {

struct RowColPlan {
    int V;        // elements per vector (16 bytes, or 1 for the scalar path)
    int nvc;      // vectors per row
    int TC, RG;   // block shape
    int gx, gy;   // grid
    int64_t chunk;  // rows per block (y)
};

constexpr int kRowsPerThread = 8;   // the unroll of the reduction's row loop
// The BN-eval backward holds a batch of dy and x rows (two vectors per row):
// eight rows took 200 VGPRs, so only two blocks fit on a CU and a stage-1
// tensor's 784 blocks ran in two rounds; four rows take 128 (every block
// resident at once; the mask-7 backward of 64 x 64 x 56 x 56 went from 31.2
// to 27.4 us, the stem-sized one unchanged).  Each thread still walks
// kRowsPerThread rows of its chunk, in two batches.
constexpr int kRowsPerThreadBn = 4;

RowColPlan plan_rowcol(int dtype, int64_t rows, int C, bool vec_ok, int target_blocks) {
    RowColPlan p;
    const int V = dtype == kBF16 ? 8 : 4;
    p.V = (vec_ok && C % V == 0) ? V : 1;   // a row must hold whole vectors
    p.nvc = std::max(C / p.V, 1);
    // at most 64 channel vectors per block: the other threads of the block
    // walk more rows of the same columns, which the block reduces in LDS, so
    // fewer partial rows reach the finalize pass
    p.TC = std::min(p.nvc, 64);
    p.RG = 256 / p.TC;
    p.gx = (p.nvc + p.TC - 1) / p.TC;
    int64_t want_y = std::max<int64_t>(1, target_blocks / p.gx);
    // at least one batch of kRowsPerThread rows per thread (all its loads in
    // flight at once), so the partials stay small next to the input
    int64_t max_y = std::max<int64_t>(1, rows / (int64_t)(p.RG * kRowsPerThread));
    p.gy = (int)std::max<int64_t>(1, std::min<int64_t>(want_y, max_y));
    p.gy = std::min(p.gy, 65535);
    p.chunk = (rows + p.gy - 1) / p.gy;
    return p;
}

bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <typename T, int V> struct VecT;
template <typename T> struct VecT<T, 1> {
    T e[1];
    __device__ __forceinline__ void load(const T *p) { e[0] = p[0]; }
    __device__ __forceinline__ void store(T *p) const { p[0] = e[0]; }
};
template <typename T> struct VecT<T, 16 / sizeof(T)> {
    union {
        u32x4 u;
        T e[16 / sizeof(T)];
    };
    __device__ __forceinline__ void load(const T *p) { u = *reinterpret_cast<const u32x4 *>(p); }
    __device__ __forceinline__ void store(T *p) const { *reinterpret_cast<u32x4 *>(p) = u; }
};

// Per-channel parameters (BN statistics, gamma, beta; any may be absent)
// read through a buffer descriptor of n elements, or of none when the array
// is absent, so a read past the end or of an absent array returns zeros and
// is issued without a branch.  Element-wise reads behind a null test each
// sat in its own branch, and every one waited for the one before.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t param_rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, p ? (int)bytes : 0, 0x00020000);
}
template <typename T>
__device__ __forceinline__ float param_at(__amdgpu_buffer_rsrc_t r, uint32_t i) {
    if constexpr (sizeof(T) == 2) return __uint_as_float((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)(i * 2), 0, 0) << 16);
    else return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)(i * 4), 0, 0));
}
// V consecutive parameters starting at element i (16 bytes when V > 1)
template <typename T, int V>
__device__ __forceinline__ void params_at(__amdgpu_buffer_rsrc_t r, uint32_t i, float (&out)[V]) {
    if constexpr (V == 1) {
        out[0] = param_at<T>(r, i);
    } else {
        VecT<T, V> v;
        v.u = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(i * sizeof(T)), 0, 0);
#pragma unroll
        for (int e = 0; e < V; ++e) out[e] = to_f32(v.e[e]);
    }
}

}  // namespace

// ---------------------------------------------------------------- BN-eval fwd
// BN-eval forward as one linear sweep: x is viewed as nvec = rows*C/V
// consecutive V-element vectors, and each thread handles U of them with all
// U loads in flight at once (the grid covers the tensor in one pass).
//  * contiguous mapping (256 % nvc == 0, nvc = vectors per row): block b
//    owns vectors [b*256*U, (b+1)*256*U) and thread t handles
//    b*256*U + u*256 + t, so a block streams one contiguous 256*U*16-byte
//    range;
//  * strided mapping (any nvc): thread i handles i + u*T (T = threads in the
//    grid, a multiple of nvc).
// Either way a thread's vectors all hold the same channels, so it folds
// (s, t) for its V channels once.
// U = kBnFlatU: 4 beat 8 and 16 on the ResNet-18-shaped stack's layers
// (stage 1, 51 MB: 12.4 against 13.2 and 13.5 us; the stack's BN-eval
// forward 165 against 169 us, alternating runs on one box).
constexpr int kBnFlatU = 4;
constexpr int kBnU = 8;   // vectors per thread of bn_nchw_kernel (below)

template <typename T, int V>
__global__ __launch_bounds__(256) void bn_fwd_flat_kernel(const T *__restrict__ x, const T *__restrict__ mean,
                                                          const T *__restrict__ var, const T *__restrict__ gamma,
                                                          const T *__restrict__ beta, float eps, int64_t nvec,
                                                          int nvc, bool contig, T *__restrict__ y) {
    const int64_t stride = contig ? 256 : (int64_t)gridDim.x * blockDim.x;
    const int64_t i0 = contig ? (int64_t)blockIdx.x * 256 * kBnFlatU + threadIdx.x
                              : (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int c0 = (int)(i0 % nvc) * V;
    VecT<T, V> pm, pv, pg, pb;
    if (mean) pm.load(mean + c0);
    pv.load(var + c0);
    if (gamma) pg.load(gamma + c0);
    if (beta) pb.load(beta + c0);
    float s[V], t[V];
#pragma unroll
    for (int e = 0; e < V; ++e) {
        const float g = gamma ? to_f32(pg.e[e]) : 1.f;
        const float b = beta ? to_f32(pb.e[e]) : 0.f;
        const float m = mean ? to_f32(pm.e[e]) : 0.f;
        s[e] = g * rsqrtf(to_f32(pv.e[e]) + eps);
        t[e] = b - m * s[e];
    }
    for (int64_t i = i0; i < nvec; i += contig ? nvec : kBnFlatU * stride) {
        VecT<T, V> v[kBnFlatU];
#pragma unroll
        for (int u = 0; u < kBnFlatU; ++u)
            if (i + u * stride < nvec) v[u].load(x + (i + u * stride) * V);
#pragma unroll
        for (int u = 0; u < kBnFlatU; ++u) {
            if (i + u * stride < nvec) {
#pragma unroll
                for (int e = 0; e < V; ++e) v[u].e[e] = from_f32<T>(fmaf(to_f32(v[u].e[e]), s[e], t[e]));
                v[u].store(y + (i + u * stride) * V);
            }
        }
    }
}

// BN-eval over a logical-NCHW tensor stored plane by plane (the plain
// row-major layout of [N, C, H, W]): vector i of V elements lies in plane
// i / vpp (vpp = HW / V vectors per plane), whose channel is plane % C.  A
// block streams 256 * kBnU consecutive vectors, each thread kBnU of them with
// all loads in flight; the per-channel scale and shift are formed per vector
// from the (cached) parameter arrays.
template <typename T, int V>
__global__ __launch_bounds__(256) void bn_nchw_kernel(const T *__restrict__ x, const T *__restrict__ mean,
                                                      const T *__restrict__ var, const T *__restrict__ gamma,
                                                      const T *__restrict__ beta, float eps, uint32_t nvec,
                                                      uint32_t vpp, uint32_t C, T *__restrict__ y) {
    const uint32_t i0 = blockIdx.x * 256u * kBnU + threadIdx.x;
    const __amdgpu_buffer_rsrc_t rm = param_rsrc(mean, C * sizeof(T)), rv = param_rsrc(var, C * sizeof(T));
    const __amdgpu_buffer_rsrc_t rg = param_rsrc(gamma, C * sizeof(T)), rb = param_rsrc(beta, C * sizeof(T));
    VecT<T, V> v[kBnU];
    float pm[kBnU], pv[kBnU], pg[kBnU], pb[kBnU];
#pragma unroll
    for (int u = 0; u < kBnU; ++u) {
        const uint32_t i = i0 + u * 256u;
        if (i < nvec) v[u].load(x + (size_t)i * V);
        const uint32_t c = ((i < nvec ? i : 0) / vpp) % C;
        pm[u] = param_at<T>(rm, c);
        pv[u] = param_at<T>(rv, c);
        pg[u] = param_at<T>(rg, c);
        pb[u] = param_at<T>(rb, c);
    }
#pragma unroll
    for (int u = 0; u < kBnU; ++u) {
        const uint32_t i = i0 + u * 256u;
        if (i >= nvec) continue;
        const float g = gamma ? pg[u] : 1.f;
        const float sc = g * rsqrtf(pv[u] + eps), sh = pb[u] - pm[u] * sc;
#pragma unroll
        for (int e = 0; e < V; ++e) v[u].e[e] = from_f32<T>(fmaf(to_f32(v[u].e[e]), sc, sh));
        v[u].store(y + (size_t)i * V);
    }
}

// One row vector of the reduction.  x comes as a value with a flag and the
// dgamma term is accumulated without a branch: a pointer to x that may be
// null, or a conditional update inside the unrolled loop, left the
// accumulators in per-lane scratch memory.
template <typename T, int V, int MODE>
__device__ __forceinline__ void rc_row(const VecT<T, V> &va, const VecT<T, V> &vx, bool use_x, T *__restrict__ dx,
                                       int64_t off, const float (&s)[V], const float (&mu)[V],
                                       const float (&inv)[V], float (&acc_b)[V], float (&acc_g)[V]) {
    if constexpr (MODE == 0) {
#pragma unroll
        for (int e = 0; e < V; ++e) acc_b[e] += to_f32(va.e[e]);
    } else {
        if (dx) {
            VecT<T, V> o;
#pragma unroll
            for (int e = 0; e < V; ++e) o.e[e] = from_f32<T>(to_f32(va.e[e]) * s[e]);
            o.store(dx + off);
        }
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const float d = to_f32(va.e[e]);
            acc_b[e] += d;
            // branch-free: acc_g is written out only when use_x
            const float xh = use_x ? (to_f32(vx.e[e]) - mu[e]) * inv[e] : 0.f;
            acc_g[e] += d * xh;
        }
    }
}

// ------------------------------------------- BN-eval bwd / column sums (partials)
// MODE 0: column sums of a (bias gradient): part0[by][c] = sum a
// MODE 1: BN-eval backward: dx = a*s (if dx), part0 = sum a*(x-mu)*inv (if want_g),
//         part1 = sum a (if want_b)
template <typename T, int V, int MODE>
__global__ __launch_bounds__(256) void rowcol_reduce_kernel(
    const T *__restrict__ a, const T *__restrict__ x, const T *__restrict__ mean,
    const T *__restrict__ var, const T *__restrict__ gamma, float eps, int64_t rows, int C, int TC,
    int RG, int64_t chunk, T *__restrict__ dx, bool want_g, bool want_b, float *__restrict__ part0,
    float *__restrict__ part1) {
    __shared__ float red[2][256 * V];
    const int tc = threadIdx.x % TC, rg = threadIdx.x / TC;
    const int cv = blockIdx.x * TC + tc;
    const bool active = rg < RG && cv * V < C;
    const int c0 = cv * V;
    float acc_g[V], acc_b[V], s[V], mu[V], inv[V];
#pragma unroll
    for (int e = 0; e < V; ++e) {
        acc_g[e] = 0.f;
        acc_b[e] = 0.f;
        s[e] = mu[e] = inv[e] = 0.f;
    }
    if (active) {
        if constexpr (MODE == 1) {
            // var is read only when dx or dgamma is requested: a beta-only
            // record does not keep the running statistics (var == nullptr).
            if (dx || want_g) {
                float pv[V], pg[V], pm[V];
                params_at<T, V>(param_rsrc(var, C * sizeof(T)), c0, pv);
                params_at<T, V>(param_rsrc(gamma, C * sizeof(T)), c0, pg);
                params_at<T, V>(param_rsrc(want_g ? mean : nullptr, C * sizeof(T)), c0, pm);
#pragma unroll
                for (int e = 0; e < V; ++e) {
                    inv[e] = 1.f / sqrtf(pv[e] + eps);
                    s[e] = (gamma ? pg[e] : 1.f) * inv[e];
                    mu[e] = pm[e];
                }
            }
        }
        const int64_t r0 = (int64_t)blockIdx.y * chunk;
        const int64_t r1 = min(rows, r0 + chunk);
        int64_t r = r0 + rg;
        constexpr int U = MODE == 1 ? kRowsPerThreadBn : kRowsPerThread;
        const bool use_x = MODE == 1 && want_g;
        for (; r + (U - 1) * RG < r1; r += U * RG) {
            VecT<T, V> va[U], vx[U] = {};
#pragma unroll
            for (int u = 0; u < U; ++u) va[u].load(a + (r + u * RG) * C + c0);
            if (use_x) {
#pragma unroll
                for (int u = 0; u < U; ++u) vx[u].load(x + (r + u * RG) * C + c0);
            }
#pragma unroll
            for (int u = 0; u < U; ++u)
                rc_row<T, V, MODE>(va[u], vx[u], use_x, dx, (r + u * RG) * C + c0, s, mu, inv, acc_b, acc_g);
        }
        for (; r < r1; r += RG) {
            VecT<T, V> va, vx = {};
            va.load(a + r * C + c0);
            if (use_x) vx.load(x + r * C + c0);
            rc_row<T, V, MODE>(va, vx, use_x, dx, r * C + c0, s, mu, inv, acc_b, acc_g);
        }
    }
    const bool need_b = MODE == 0 || want_b;
    const bool need_g = MODE == 1 && want_g;
    if (!need_b && !need_g) return;   // uniform over the block
    // Combine the row groups in a fixed order.  With TC a power of two
    // (every vectorized channel count that is a multiple of 8 or 16 up to
    // 512 channels per block column) first inside each wave, by butterfly
    // shuffles over the lanes that share a channel vector (lane = rg * TC +
    // tc, so they are TC apart), then the four waves' sums through LDS.
    // Otherwise through LDS, one thread per (channel vector, element) adding
    // the row groups in order.  (The first version let TC threads add all
    // RG * V sums serially out of LDS: a tail of several microseconds per
    // block that dominated the smaller tensors.)
    const int64_t orow = (int64_t)blockIdx.y * C;
    auto put = [&](int c, float sb, float sg) {
        if (MODE == 0) {
            part0[orow + c] = sb;
        } else {
            if (need_g) part0[orow + c] = sg;
            if (want_b) part1[orow + c] = sb;
        }
    };
    if ((TC & (TC - 1)) == 0) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        for (int off = TC; off < 64; off <<= 1) {
#pragma unroll
            for (int e = 0; e < V; ++e) {
                acc_b[e] += __shfl_xor(acc_b[e], off);
                if (MODE == 1) acc_g[e] += __shfl_xor(acc_g[e], off);
            }
        }
        // lanes 0 .. TC-1 of each wave now hold the wave's sums for tc = lane
        if (lane < TC) {
#pragma unroll
            for (int e = 0; e < V; ++e) {
                red[0][(wave * TC + lane) * V + e] = acc_b[e];
                red[1][(wave * TC + lane) * V + e] = acc_g[e];
            }
        }
        __syncthreads();
        if (threadIdx.x < TC && cv * V < C) {
#pragma unroll
            for (int e = 0; e < V; ++e) {
                float sb = 0.f, sg = 0.f;
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    sb += red[0][(w * TC + tc) * V + e];
                    sg += red[1][(w * TC + tc) * V + e];
                }
                put(c0 + e, sb, sg);
            }
        }
    } else {
#pragma unroll
        for (int e = 0; e < V; ++e) {
            red[0][threadIdx.x * V + e] = acc_b[e];
            red[1][threadIdx.x * V + e] = acc_g[e];
        }
        __syncthreads();
        for (int j = threadIdx.x; j < TC * V; j += 256) {
            const int tcj = j / V, e = j - tcj * V;
            const int c = (blockIdx.x * TC + tcj) * V + e;
            if (c >= C) continue;
            float sb = 0.f, sg = 0.f;
            for (int q = 0; q < RG; ++q) {
                sb += red[0][(q * TC + tcj) * V + e];
                sg += red[1][(q * TC + tcj) * V + e];
            }
            put(c, sb, sg);
        }
    }
}

// out[c] = sum_y part[y][c], rounded once to T, for up to two (part, out)
// pairs (grid y).  A block owns 4 columns; its 64 thread rows split the
// partial rows, each issuing 16 loads at once (one memory round trip per
// 1024 partial rows), and meet in LDS in a fixed tree order.
template <typename T>
__global__ __launch_bounds__(256) void finalize_kernel(const float *__restrict__ part0, T *__restrict__ out0,
                                                       const float *__restrict__ part1, T *__restrict__ out1, int gy,
                                                       int C) {
    __shared__ float red[64][5];
    const float *__restrict__ part = blockIdx.y ? part1 : part0;
    T *__restrict__ out = blockIdx.y ? out1 : out0;
    const int cl = threadIdx.x & 3, yg = threadIdx.x >> 2;
    const int c = blockIdx.x * 4 + cl;
    float s = 0.f;
    if (c < C) {
        for (int y0 = yg; y0 < gy; y0 += 64 * 16) {
            float a[16];
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                const int y = y0 + 64 * k;
                a[k] = y < gy ? part[(int64_t)y * C + c] : 0.f;
            }
#pragma unroll
            for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
                for (int k = 0; k < w; ++k) a[k] += a[k + w];
            s += a[0];
        }
    }
    red[yg][cl] = s;
    __syncthreads();
    for (int off = 32; off >= 1; off >>= 1) {
        if (yg < off) red[yg][cl] += red[yg + off][cl];
        __syncthreads();
    }
    if (yg == 0 && c < C) out[c] = from_f32<T>(red[0][cl]);
}

// ---------------------------------------------------------------- avgpool
// y[n][c] = (1/L) sum_l x[n][l][c]; grid (column tiles, N)
template <typename T, int V>
__global__ __launch_bounds__(256) void avgpool_fwd_kernel(const T *__restrict__ x, int L, int C, int TC,
                                                          int RG, T *__restrict__ y) {
    __shared__ float red[256 * V];
    const int tc = threadIdx.x % TC, rg = threadIdx.x / TC;
    const int cv = blockIdx.x * TC + tc;
    const bool active = rg < RG && cv * V < C;
    const int c0 = cv * V;
    const int n = blockIdx.y;
    float acc[V];
#pragma unroll
    for (int e = 0; e < V; ++e) acc[e] = 0.f;
    if (active) {
        for (int l = rg; l < L; l += RG) {
            VecT<T, V> v;
            v.load(x + ((int64_t)n * L + l) * C + c0);
#pragma unroll
            for (int e = 0; e < V; ++e) acc[e] += to_f32(v.e[e]);
        }
    }
#pragma unroll
    for (int e = 0; e < V; ++e) red[threadIdx.x * V + e] = acc[e];
    __syncthreads();
    if (rg == 0 && active) {
        VecT<T, V> o;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            float s = 0.f;
            for (int q = 0; q < RG; ++q) s += red[(q * TC + tc) * V + e];
            o.e[e] = from_f32<T>(s / (float)L);
        }
        o.store(y + (int64_t)n * C + c0);
    }
}

// dx[n][l][c] = dy[n][c] / L
template <typename T, int V>
__global__ __launch_bounds__(256) void avgpool_bwd_kernel(const T *__restrict__ dy, int N, int L, int C,
                                                          T *__restrict__ dx) {
    const int nvc = C / V;
    const int64_t total = (int64_t)N * L * nvc;
    const float invL = 1.f / (float)L;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int cv = (int)(i % nvc);
        const int64_t pix = i / nvc;
        const int n = (int)(pix / L);
        VecT<T, V> v;
        v.load(dy + (int64_t)n * C + cv * V);
#pragma unroll
        for (int e = 0; e < V; ++e) v.e[e] = from_f32<T>(to_f32(v.e[e]) * invL);
        v.store(dx + pix * C + cv * V);
    }
}

// ------------------------------------------------------------------ launchers
namespace {
constexpr int kTargetBlocks = 1024;

template <typename T, int V, int MODE>
int reduce_t(const RowColPlan &p, const void *a, const void *x, const void *mean, const void *var,
             const void *gamma, float eps, int64_t rows, int C, void *dx, bool want_g, bool want_b,
             float *part0, float *part1, hipStream_t st) {
    hipLaunchKernelGGL((rowcol_reduce_kernel<T, V, MODE>), dim3(p.gx, p.gy), dim3(256), 0, st,
                       (const T *)a, (const T *)x, (const T *)mean, (const T *)var, (const T *)gamma, eps,
                       rows, C, p.TC, p.RG, p.chunk, (T *)dx, want_g, want_b, part0, part1);
    return (int)hipGetLastError();
}

// One launch for one or two column reductions (part1 / out1 may be null).
template <typename T>
int finalize_t(const float *part0, void *out0, const float *part1, void *out1, int gy, int C, hipStream_t st) {
    hipLaunchKernelGGL(finalize_kernel<T>, dim3((C + 3) / 4, out1 ? 2 : 1), dim3(256), 0, st, part0, (T *)out0, part1,
                       (T *)out1, gy, C);
    return (int)hipGetLastError();
}

int finalize(int dtype, const float *part0, void *out0, const float *part1, void *out1, int gy, int C,
             hipStream_t st) {
    return dtype == kBF16 ? finalize_t<bf16>(part0, out0, part1, out1, gy, C, st)
                          : finalize_t<float>(part0, out0, part1, out1, gy, C, st);
}

}  // namespace

namespace {
// The flat per-channel sweep y = x * s_c + t_c; `pk` is the profiling kind
// its launch counts as (the BN forward, or a BN backward that wants dx only).
int bn_sweep(int dtype, const void *x, const void *mean, const void *var, const void *gamma, const void *beta,
             float eps, int64_t rows, int C, void *y, void *stream, unsigned pk) {
    if (rows == 0 || C == 0) return 0;
    const int V = dtype == kBF16 ? 8 : 4;
    // 16-byte vectors of x, y and of the per-channel parameters
    const bool vec = C % V == 0 && al16(x) && al16(y) && al16(mean) && al16(var) &&
                     (!gamma || al16(gamma)) && (!beta || al16(beta));
    const int Ve = vec ? V : 1;
    const int nvc = C / Ve;
    const int64_t nvec = rows * (int64_t)nvc;
    // one pass of kBnFlatU vectors per thread; the thread count is rounded up to
    // a multiple of nvc (block granularity q) so every thread keeps its
    // channels
    int64_t q = 1;
    {
        int64_t a = nvc, b = 256;
        while (b) { const int64_t r = a % b; a = b; b = r; }
        q = nvc / a;   // nvc / gcd(nvc, 256)
    }
    int64_t blocks = std::max<int64_t>(1, (nvec + 256 * kBnFlatU - 1) / (256 * kBnFlatU));
    const bool contig = 256 % nvc == 0;
    if (!contig) blocks = (blocks + q - 1) / q * q;
    hipStream_t st = (hipStream_t)stream;
    prof_mark(pk, st, true);
    if (dtype == kBF16) {
        if (vec)
            hipLaunchKernelGGL((bn_fwd_flat_kernel<bf16, 8>), dim3((unsigned)blocks), dim3(256), 0, st, (const bf16 *)x,
                               (const bf16 *)mean, (const bf16 *)var, (const bf16 *)gamma, (const bf16 *)beta, eps, nvec,
                               nvc, contig, (bf16 *)y);
        else
            hipLaunchKernelGGL((bn_fwd_flat_kernel<bf16, 1>), dim3((unsigned)blocks), dim3(256), 0, st, (const bf16 *)x,
                               (const bf16 *)mean, (const bf16 *)var, (const bf16 *)gamma, (const bf16 *)beta, eps, nvec,
                               nvc, contig, (bf16 *)y);
    } else {
        if (vec)
            hipLaunchKernelGGL((bn_fwd_flat_kernel<float, 4>), dim3((unsigned)blocks), dim3(256), 0, st, (const float *)x,
                               (const float *)mean, (const float *)var, (const float *)gamma, (const float *)beta, eps,
                               nvec, nvc, contig, (float *)y);
        else
            hipLaunchKernelGGL((bn_fwd_flat_kernel<float, 1>), dim3((unsigned)blocks), dim3(256), 0, st, (const float *)x,
                               (const float *)mean, (const float *)var, (const float *)gamma, (const float *)beta, eps,
                               nvec, nvc, contig, (float *)y);
    }
    const int err = (int)hipGetLastError();
    prof_mark(pk, st, false);
    return err;
}
}  // namespace

int launch_bn_fwd(int dtype, const void *x, const void *mean, const void *var, const void *gamma,
                  const void *beta, float eps, int64_t rows, int C, void *y, void *stream) {
    return bn_sweep(dtype, x, mean, var, gamma, beta, eps, rows, C, y, stream, kProfBn);
}

int launch_bn_nchw(int dtype, const void *x, const void *mean, const void *var, const void *gamma, const void *beta,
                   float eps, int64_t N, int C, int64_t HW, void *y, void *stream, bool backward) {
    const int64_t n = N * C * HW;
    if (n == 0) return 0;
    const int V = dtype == kBF16 ? 8 : 4;
    const bool vec = HW % V == 0 && al16(x) && al16(y);
    const int Ve = vec ? V : 1;
    const int64_t nvec = n / Ve;
    const unsigned blocks = (unsigned)((nvec + 256 * kBnU - 1) / (256 * kBnU));
    hipStream_t st = (hipStream_t)stream;
    const unsigned pk = backward ? kProfRed : kProfBn;
    prof_mark(pk, st, true);
    const uint32_t vpp = (uint32_t)(HW / Ve);
    if (dtype == kBF16) {
        if (vec) hipLaunchKernelGGL((bn_nchw_kernel<bf16, 8>), dim3(blocks), dim3(256), 0, st, (const bf16 *)x, (const bf16 *)mean,
                                    (const bf16 *)var, (const bf16 *)gamma, (const bf16 *)beta, eps, (uint32_t)nvec, vpp,
                                    (uint32_t)C, (bf16 *)y);
        else hipLaunchKernelGGL((bn_nchw_kernel<bf16, 1>), dim3(blocks), dim3(256), 0, st, (const bf16 *)x, (const bf16 *)mean,
                                (const bf16 *)var, (const bf16 *)gamma, (const bf16 *)beta, eps, (uint32_t)nvec, vpp,
                                (uint32_t)C, (bf16 *)y);
    } else {
        if (vec) hipLaunchKernelGGL((bn_nchw_kernel<float, 4>), dim3(blocks), dim3(256), 0, st, (const float *)x,
                                    (const float *)mean, (const float *)var, (const float *)gamma, (const float *)beta, eps,
                                    (uint32_t)nvec, vpp, (uint32_t)C, (float *)y);
        else hipLaunchKernelGGL((bn_nchw_kernel<float, 1>), dim3(blocks), dim3(256), 0, st, (const float *)x,
                                (const float *)mean, (const float *)var, (const float *)gamma, (const float *)beta, eps,
                                (uint32_t)nvec, vpp, (uint32_t)C, (float *)y);
    }
    const int err = (int)hipGetLastError();
    prof_mark(pk, st, false);
    return err;
}

static RowColPlan bn_bwd_plan(int dtype, int64_t rows, int C, bool vec) {
    return plan_rowcol(dtype, rows, C, vec, kTargetBlocks);
}

size_t bn_bwd_workspace(int dtype, int64_t rows, int C) {
    // sized for the scalar plan too (it can only have more row chunks)
    RowColPlan p1 = bn_bwd_plan(dtype, rows, C, true), p0 = bn_bwd_plan(dtype, rows, C, false);
    const int gy = std::max(p1.gy, p0.gy);
    return (size_t)2 * gy * C * sizeof(float);
}

int launch_bn_bwd(int dtype, const void *dy, const void *x, const void *mean, const void *var,
                  const void *gamma, float eps, int64_t rows, int C, void *dx, void *dgamma, void *dbeta,
                  void *ws, void *stream) {
    if (C == 0) return 0;
    // pointers the requested outputs need (the host runtime guarantees them)
    if ((dx || dgamma) && !var) return (int)hipErrorInvalidValue;
    if (dgamma && (!x || !mean)) return (int)hipErrorInvalidValue;
    // dx alone (frozen gamma and beta) is the forward's per-channel sweep
    // with a zero mean and no shift: dx = dy * gamma / sqrt(var + eps)
    if (dx && !dgamma && !dbeta) return bn_sweep(dtype, dy, nullptr, var, gamma, nullptr, eps, rows, C, dx, stream, kProfRed);
    hipStream_t st = (hipStream_t)stream;
    prof_mark(kProfRed, st, true);
    const int V = dtype == kBF16 ? 8 : 4;
    const bool vec = C % V == 0 && al16(dy) && (!x || al16(x)) && (!dx || al16(dx));
    RowColPlan p = bn_bwd_plan(dtype, rows, C, vec);
    const bool want_g = dgamma != nullptr, want_b = dbeta != nullptr;
    float *part0 = static_cast<float *>(ws);
    float *part1 = part0 + (size_t)p.gy * C;
    if (rows > 0) {
        int err;
        if (dtype == kBF16)
            err = vec ? reduce_t<bf16, 8, 1>(p, dy, x, mean, var, gamma, eps, rows, C, dx, want_g, want_b, part0, part1, st)
                      : reduce_t<bf16, 1, 1>(p, dy, x, mean, var, gamma, eps, rows, C, dx, want_g, want_b, part0, part1, st);
        else
            err = vec ? reduce_t<float, 4, 1>(p, dy, x, mean, var, gamma, eps, rows, C, dx, want_g, want_b, part0, part1, st)
                      : reduce_t<float, 1, 1>(p, dy, x, mean, var, gamma, eps, rows, C, dx, want_g, want_b, part0, part1, st);
        if (err) return err;
    }
    const int gy = rows > 0 ? p.gy : 0;
    if (want_g || want_b) {
        // dgamma and dbeta in one finalize launch
        const int err = want_g ? finalize(dtype, part0, dgamma, want_b ? part1 : nullptr, dbeta, gy, C, st)
                               : finalize(dtype, part1, dbeta, nullptr, nullptr, gy, C, st);
        if (err) return err;
    }
    prof_mark(kProfRed, st, false);
    return 0;
}

size_t colsum_workspace(int dtype, int64_t rows, int C) {
    RowColPlan p1 = plan_rowcol(dtype, rows, C, true, kTargetBlocks);
    RowColPlan p0 = plan_rowcol(dtype, rows, C, false, kTargetBlocks);
    return (size_t)std::max(p1.gy, p0.gy) * C * sizeof(float);
}

int launch_colsum_finalize(int dtype, const float *part, int rows, int cols, void *out, void *stream) {
    if (cols == 0) return 0;
    prof_mark(kProfRed, stream, true);
    const int err = finalize(dtype, part, out, nullptr, nullptr, rows, cols, (hipStream_t)stream);
    prof_mark(kProfRed, stream, false);
    return err;
}

int launch_colsum(int dtype, const void *in, int64_t rows, int C, void *out, void *ws, void *stream) {
    if (C == 0) return 0;
    hipStream_t st = (hipStream_t)stream;
    const int V = dtype == kBF16 ? 8 : 4;
    const bool vec = C % V == 0 && al16(in);
    RowColPlan p = plan_rowcol(dtype, rows, C, vec, kTargetBlocks);
    float *part = static_cast<float *>(ws);
    prof_mark(kProfRed, st, true);
    if (rows > 0) {
        int err;
        if (dtype == kBF16)
            err = vec ? reduce_t<bf16, 8, 0>(p, in, nullptr, nullptr, nullptr, nullptr, 0.f, rows, C, nullptr, false, true, part, nullptr, st)
                      : reduce_t<bf16, 1, 0>(p, in, nullptr, nullptr, nullptr, nullptr, 0.f, rows, C, nullptr, false, true, part, nullptr, st);
        else
            err = vec ? reduce_t<float, 4, 0>(p, in, nullptr, nullptr, nullptr, nullptr, 0.f, rows, C, nullptr, false, true, part, nullptr, st)
                      : reduce_t<float, 1, 0>(p, in, nullptr, nullptr, nullptr, nullptr, 0.f, rows, C, nullptr, false, true, part, nullptr, st);
        if (err) return err;
    }
    const int err = finalize(dtype, part, out, nullptr, nullptr, rows > 0 ? p.gy : 0, C, st);
    prof_mark(kProfRed, st, false);
    return err;
}

int launch_avgpool_fwd(int dtype, const void *x, int N, int L, int C, void *y, void *stream) {
    if (N == 0 || C == 0) return 0;
    hipStream_t st = (hipStream_t)stream;
    const int V = dtype == kBF16 ? 8 : 4;
    const bool vec = C % V == 0 && al16(x) && al16(y);
    const int v = vec ? V : 1;
    const int nvc = C / v;
    const int TC = std::min(nvc, 256), RG = 256 / TC;
    dim3 grid((nvc + TC - 1) / TC, N);
    if (dtype == kBF16) {
        if (vec) hipLaunchKernelGGL((avgpool_fwd_kernel<bf16, 8>), grid, dim3(256), 0, st, (const bf16 *)x, L, C, TC, RG, (bf16 *)y);
        else hipLaunchKernelGGL((avgpool_fwd_kernel<bf16, 1>), grid, dim3(256), 0, st, (const bf16 *)x, L, C, TC, RG, (bf16 *)y);
    } else {
        if (vec) hipLaunchKernelGGL((avgpool_fwd_kernel<float, 4>), grid, dim3(256), 0, st, (const float *)x, L, C, TC, RG, (float *)y);
        else hipLaunchKernelGGL((avgpool_fwd_kernel<float, 1>), grid, dim3(256), 0, st, (const float *)x, L, C, TC, RG, (float *)y);
    }
    return (int)hipGetLastError();
}

int launch_avgpool_bwd(int dtype, const void *dy, int N, int L, int C, void *dx, void *stream) {
    if (N == 0 || C == 0 || L == 0) return 0;
    hipStream_t st = (hipStream_t)stream;
    const int V = dtype == kBF16 ? 8 : 4;
    const bool vec = C % V == 0 && al16(dy) && al16(dx);
    const int64_t total = (int64_t)N * L * (C / (vec ? V : 1));
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
    if (dtype == kBF16) {
        if (vec) hipLaunchKernelGGL((avgpool_bwd_kernel<bf16, 8>), dim3(blocks), dim3(256), 0, st, (const bf16 *)dy, N, L, C, (bf16 *)dx);
        else hipLaunchKernelGGL((avgpool_bwd_kernel<bf16, 1>), dim3(blocks), dim3(256), 0, st, (const bf16 *)dy, N, L, C, (bf16 *)dx);
    } else {
        if (vec) hipLaunchKernelGGL((avgpool_bwd_kernel<float, 4>), dim3(blocks), dim3(256), 0, st, (const float *)dy, N, L, C, (float *)dx);
        else hipLaunchKernelGGL((avgpool_bwd_kernel<float, 1>), dim3(blocks), dim3(256), 0, st, (const float *)dy, N, L, C, (float *)dx);
    }
    return (int)hipGetLastError();
}

}  // namespace ms

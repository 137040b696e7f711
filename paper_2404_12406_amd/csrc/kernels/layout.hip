// Strided copies between a caller's tensor layout and the dense
// channels-last layout the layer kernels read (NHWC activations, KRSC
// filters, row-major matrices).  A layer call whose tensors are in another
// layout -- NCHW, a strided slice, a transposed view -- runs its kernels on
// staged copies in transient workspace; the staging moves every byte once in
// and once out, HBM-bound.
//
// A copy is described over a 4-D index space with each side's own element
// strides.  When the unit-stride dimension of the destination differs from
// the source's (NCHW <-> NHWC: w against c), 64 x 64 tiles over those two
// dimensions pass through LDS, so that the reads run along the source's unit
// stride and the writes along the destination's; the other two dimensions
// index the tiles' batch.  Otherwise (the same fastest dimension on both
// sides, e.g. a channel slice) elements are copied in the order of that
// dimension, coalesced on both sides.
#include "common.h"

#include <algorithm>

#include "../device.h"

namespace ms {

namespace {

struct Copy4 {
    int64_t ext[4];
    int64_t ss[4], ds[4];
    int ia, ib;        // tiled path: the destination's and the source's unit-stride dims
    int o0, o1;        // tiled path: the batch dims (o1 varies fastest)
    int64_t ta, tb;    // tiled path: tiles along ia and ib
    int p[4];          // flat path: dims from fastest to slowest
};

constexpr int kT = 64;   // tile edge

// Raw vector of B bytes (B = 4, 8 or 16).
template <int B> struct Raw;
template <> struct Raw<4> { typedef uint32_t type; };
template <> struct Raw<8> { typedef uint64_t type; };
template <> struct Raw<16> { typedef u32x4 type; };

// RB / WB: bytes per access of a source row (along ib) / destination row
// (along ia); 0 = element by element.  The caller checked unit stride,
// extent and alignment for the vector widths it picked.
template <typename T, int RB, int WB>
__global__ __launch_bounds__(256) void copy4_tiled_kernel(const T *__restrict__ src, T *__restrict__ dst, const Copy4 c) {
    constexpr int PITCH = kT + 16 / (int)sizeof(T);   // 16-byte aligned rows, shifted banks
    __shared__ __attribute__((aligned(16))) T tile[kT][PITCH];
    int64_t blk = blockIdx.x;
    const int64_t tbi = blk % c.tb;
    blk /= c.tb;
    const int64_t tai = blk % c.ta;
    const int64_t bat = blk / c.ta;
    const int64_t j1 = bat % c.ext[c.o1], j0 = bat / c.ext[c.o1];
    const int64_t sbase = j0 * c.ss[c.o0] + j1 * c.ss[c.o1];
    const int64_t dbase = j0 * c.ds[c.o0] + j1 * c.ds[c.o1];
    const int64_t a0 = tai * kT, b0 = tbi * kT;
    const int64_t ea = c.ext[c.ia], eb = c.ext[c.ib];
    const int t = threadIdx.x;
    // read along the source's unit stride: tile[a][b]
    if constexpr (RB > 0) {
        typedef typename Raw<RB>::type V;
        constexpr int E = RB / (int)sizeof(T), VPR = kT / E, RPP = 256 / VPR;   // rows per pass
        const int cv = t % VPR;
        for (int r = t / VPR; r < kT; r += RPP) {
            const int64_t a = a0 + r, b = b0 + cv * E;
            if (a < ea && b < eb)
                *reinterpret_cast<V *>(&tile[r][cv * E]) = *reinterpret_cast<const V *>(src + sbase + a * c.ss[c.ia] + b);
        }
    } else {
        const int lx = t & (kT - 1);
        for (int r = t >> 6; r < kT; r += 4) {
            const int64_t a = a0 + r, b = b0 + lx;
            if (a < ea && b < eb) tile[r][lx] = src[sbase + a * c.ss[c.ia] + b * c.ss[c.ib]];
        }
    }
    __syncthreads();
    // write along the destination's unit stride
    if constexpr (WB > 0) {
        typedef typename Raw<WB>::type V;
        constexpr int E = WB / (int)sizeof(T), VPR = kT / E, RPP = 256 / VPR;
        const int av = t % VPR;
        for (int r = t / VPR; r < kT; r += RPP) {
            const int64_t a = a0 + av * E, b = b0 + r;
            if (a < ea && b < eb) {
                union {
                    V v;
                    T e[E];
                } u;
#pragma unroll
                for (int e = 0; e < E; ++e) u.e[e] = tile[av * E + e][r];
                *reinterpret_cast<V *>(dst + dbase + b * c.ds[c.ib] + a) = u.v;
            }
        }
    } else {
        const int lx = t & (kT - 1);
        for (int r = t >> 6; r < kT; r += 4) {
            const int64_t a = a0 + lx, b = b0 + r;
            if (a < ea && b < eb) dst[dbase + a * c.ds[c.ia] + b * c.ds[c.ib]] = tile[lx][r];
        }
    }
}

template <typename T, int RB>
int launch_tiled(int wb, const T *src, T *dst, const Copy4 &c, dim3 grid, hipStream_t st) {
    switch (wb) {
    case 16: hipLaunchKernelGGL((copy4_tiled_kernel<T, RB, 16>), grid, dim3(256), 0, st, src, dst, c); break;
    case 8: hipLaunchKernelGGL((copy4_tiled_kernel<T, RB, 8>), grid, dim3(256), 0, st, src, dst, c); break;
    case 4: hipLaunchKernelGGL((copy4_tiled_kernel<T, RB, (sizeof(T) <= 4 ? 4 : 0)>), grid, dim3(256), 0, st, src, dst, c); break;
    default: hipLaunchKernelGGL((copy4_tiled_kernel<T, RB, 0>), grid, dim3(256), 0, st, src, dst, c); break;
    }
    return (int)hipGetLastError();
}

template <typename T>
__global__ __launch_bounds__(256) void copy4_flat_kernel(const T *__restrict__ src, T *__restrict__ dst, const Copy4 c,
                                                         int64_t total) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total; i += (int64_t)gridDim.x * 256) {
        int64_t r = i, so = 0, dso = 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int d = c.p[k];
            const int64_t e = c.ext[d];
            const int64_t idx = r % e;
            r /= e;
            so += idx * c.ss[d];
            dso += idx * c.ds[d];
        }
        dst[dso] = src[so];
    }
}

template <typename T>
int copy4(const T *src, T *dst, Copy4 c, hipStream_t st) {
    int64_t total = 1;
    for (int d = 0; d < 4; ++d) total *= c.ext[d];
    if (total == 0) return 0;
    // unit-stride (smallest-stride) dims of each side among the dims that vary
    int ia = -1, ib = -1;
    for (int d = 0; d < 4; ++d) {
        if (c.ext[d] <= 1) continue;
        if (ia < 0 || c.ds[d] < c.ds[ia]) ia = d;
        if (ib < 0 || c.ss[d] < c.ss[ib]) ib = d;
    }
    if (ia >= 0 && ib >= 0 && ia != ib && c.ext[ia] * c.ext[ib] >= 1024) {
        c.ia = ia;
        c.ib = ib;
        int o[2], k = 0;
        for (int d = 0; d < 4; ++d)
            if (d != ia && d != ib) o[k++] = d;
        // the batch's faster dim: the one with the smaller destination stride
        c.o0 = c.ds[o[0]] >= c.ds[o[1]] ? o[0] : o[1];
        c.o1 = c.o0 == o[0] ? o[1] : o[0];
        c.ta = (c.ext[ia] + kT - 1) / kT;
        c.tb = (c.ext[ib] + kT - 1) / kT;
        const int64_t blocks = c.ta * c.tb * c.ext[c.o0] * c.ext[c.o1];
        if (blocks > INT32_MAX) return (int)hipErrorInvalidValue;
        // the widest vector (16, 8 or 4 bytes) that a side's unit-stride
        // dim allows: its extent and every other stride of the side whole
        // vectors, the base aligned to one
        auto width = [&](const int64_t *str, int unit, const void *p) {
            if (str[unit] != 1) return 0;
            for (int B = 16; B >= 4; B /= 2) {
                const int E = B / (int)sizeof(T);
                if (E < 2 || reinterpret_cast<uintptr_t>(p) % B != 0 || c.ext[unit] % E != 0) continue;
                bool ok = true;
                for (int d = 0; d < 4; ++d)
                    if (d != unit && c.ext[d] > 1 && str[d] % E != 0) ok = false;
                if (ok) return B;
            }
            return 0;
        };
        const int rb = width(c.ss, ib, src), wb = width(c.ds, ia, dst);
        const dim3 grid((unsigned)blocks);
        switch (rb) {
        case 16: return launch_tiled<T, 16>(wb, src, dst, c, grid, st);
        case 8: return launch_tiled<T, 8>(wb, src, dst, c, grid, st);
        case 4: return launch_tiled<T, (sizeof(T) <= 2 ? 4 : 0)>(wb, src, dst, c, grid, st);
        default: return launch_tiled<T, 0>(wb, src, dst, c, grid, st);
        }
    }
    // flat: destination's fastest dim first, the rest by decreasing stride order
    int p[4] = {0, 1, 2, 3};
    std::sort(p, p + 4, [&](int a, int b) { return c.ds[a] < c.ds[b] || (c.ds[a] == c.ds[b] && a > b); });
    for (int k = 0; k < 4; ++k) c.p[k] = p[k];
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 65536);
    hipLaunchKernelGGL(copy4_flat_kernel<T>, dim3(blocks), dim3(256), 0, st, src, dst, c, total);
    return (int)hipGetLastError();
}

// Dimensions a and b are one dimension on both sides when a step of a lands
// where a walk over all of b ends: s[a] == s[b] * ext[b] for the source and
// the destination strides alike.  Merging them (extent ext[a] * ext[b], b's
// strides) leaves the same element map in fewer dimensions: the H x W plane
// of an NCHW <-> NHWC copy becomes one dimension, and the tiled path gets
// whole 64 x 64 tiles instead of 64 x W ones (a 28-wide plane left more than
// half of every tile empty).
void merge_dims(Copy4 &c) {
    for (bool changed = true; changed;) {
        changed = false;
        for (int a = 0; a < 4 && !changed; ++a) {
            if (c.ext[a] <= 1) continue;
            for (int b = 0; b < 4; ++b) {
                if (b == a || c.ext[b] <= 1) continue;
                if (c.ss[a] == c.ss[b] * c.ext[b] && c.ds[a] == c.ds[b] * c.ext[b]) {
                    c.ext[b] *= c.ext[a];
                    c.ext[a] = 1;
                    changed = true;
                    break;
                }
            }
        }
    }
}

}  // namespace

int launch_copy4(int dtype, const void *src, const int64_t ext[4], const int64_t sstride[4], void *dst,
                 const int64_t dstride[4], void *stream) {
    Copy4 c{};
    for (int d = 0; d < 4; ++d) {
        c.ext[d] = ext[d];
        c.ss[d] = sstride[d];
        c.ds[d] = dstride[d];
    }
    merge_dims(c);
    hipStream_t st = (hipStream_t)stream;
    return dtype == kBF16 ? copy4(static_cast<const bf16 *>(src), static_cast<bf16 *>(dst), c, st)
                          : copy4(static_cast<const float *>(src), static_cast<float *>(dst), c, st);
}

}  // namespace ms

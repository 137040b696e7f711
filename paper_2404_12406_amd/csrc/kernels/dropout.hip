// Dropout whose backward draws its mask again (Sec. 2.2.2 of the paper): a
// stored mask, like a stored output, would keep activation memory alive for
// the backward pass; the layer keeps the state of a counter-based generator
// instead and pays for a second draw.
//
// Generator: Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw,
// "Parallel random numbers: as easy as 1, 2, 3", SC 2011).  A block maps a
// 128-bit counter and a 64-bit key to four 32-bit words; each round takes
// the 64-bit products of counter words 0 and 2 with two fixed multipliers,
// xors their high halves into words 1 and 3 and the key, and the key is
// advanced by two Weyl constants between rounds.
//
// Stream of a call: element i (memory order) takes word i mod 4 of the block
// with counter (b mod 2^32, b div 2^32, 0, 0), b = offset + floor(i / 4), and
// key (seed mod 2^32, seed div 2^32); it is kept iff that word is >= thresh.
//
//   out_i = in_i * (kept ? scale : 0)     (forward: in = x; backward: in = dy)
//   drop_all (p = 1): out_i = 0
//
// Forward and backward are the same pass.  A thread owns groups of 8
// consecutive elements (one 16-byte vector of bf16, two of fp32) -- two
// generator blocks -- and keeps kU groups' loads in flight.  HBM bytes per
// element: 2 * elt; ALU work per element: a quarter of a 10-round block.
#include <algorithm>

#include "common.h"
#include "../device.h"

namespace ms {
namespace {

constexpr uint32_t kMul0 = 0xD2511F53u, kMul1 = 0xCD9E8D57u;     // round multipliers
constexpr uint32_t kWeyl0 = 0x9E3779B9u, kWeyl1 = 0xBB67AE85u;   // key increments
constexpr int kU = 2;   // groups per thread per pass

struct Words {
    uint32_t w[4];
};

// One generator block for counter (c0, c1, 0, 0) under key (k0, k1).
__device__ __forceinline__ Words philox_block(uint32_t c0, uint32_t c1, uint32_t k0, uint32_t k1) {
    uint32_t c2 = 0u, c3 = 0u;
#pragma unroll
    for (int round = 0; round < 10; ++round) {
        const uint64_t p0 = (uint64_t)kMul0 * c0, p1 = (uint64_t)kMul1 * c2;   // one 32 x 32 -> 64 multiply each
        const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
        const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
        const uint32_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
        c0 = n0;
        c1 = lo1;
        c2 = n2;
        c3 = lo0;
        k0 += kWeyl0;
        k1 += kWeyl1;
    }
    return Words{{c0, c1, c2, c3}};
}

template <typename T, bool VEC>
__global__ __launch_bounds__(256) void dropout_kernel(const T *__restrict__ in, T *__restrict__ out, int64_t n,
                                                      int64_t ngroups, uint32_t k0, uint32_t k1, uint64_t offset,
                                                      uint32_t thresh, float scale, int drop_all) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t v0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; v0 < ngroups; v0 += kU * stride) {
        Group8<T> g[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u)
            if (v0 + u * stride < ngroups) g[u] = load_group8<T, VEC>(in, (v0 + u * stride) * 8, n);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int64_t v = v0 + u * stride;
            if (v >= ngroups) continue;
            const uint64_t b = offset + 2u * (uint64_t)v;
            const Words r0 = philox_block((uint32_t)b, (uint32_t)(b >> 32), k0, k1);
            const Words r1 = philox_block((uint32_t)(b + 1u), (uint32_t)((b + 1u) >> 32), k0, k1);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const uint32_t w = e < 4 ? r0.w[e] : r1.w[e - 4];
                const float s = w >= thresh ? scale : 0.f;
                g[u].e[e] = drop_all ? (T)0.f : from_f32<T>(to_f32(g[u].e[e]) * s);
            }
            store_group8<T, VEC>(out, v * 8, n, g[u]);
        }
    }
}

bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <typename T>
int run(const void *in, int64_t n, void *out, uint64_t seed, uint64_t offset, uint32_t thresh, float scale,
        int drop_all, hipStream_t st) {
    const int64_t ng = (n + 7) / 8;
    const int grid = (int)std::max<int64_t>(1, std::min<int64_t>((ng + 256 * kU - 1) / (256 * kU), 65536));
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    if (al16(in) && al16(out))
        hipLaunchKernelGGL((dropout_kernel<T, true>), dim3(grid), dim3(256), 0, st, (const T *)in, (T *)out, n, ng,
                           k0, k1, offset, thresh, scale, drop_all);
    else
        hipLaunchKernelGGL((dropout_kernel<T, false>), dim3(grid), dim3(256), 0, st, (const T *)in, (T *)out, n, ng,
                           k0, k1, offset, thresh, scale, drop_all);
    return (int)hipGetLastError();
}

}  // namespace

int launch_dropout(int dtype, const void *in, int64_t n, void *out, uint64_t seed, uint64_t offset, uint32_t thresh,
                   float scale, int drop_all, void *stream) {
    if (n == 0) return 0;
    hipStream_t st = (hipStream_t)stream;
    prof_mark(kProfAct, st, true);
    const int err = dtype == kBF16 ? run<bf16>(in, n, out, seed, offset, thresh, scale, drop_all, st)
                                   : run<float>(in, n, out, seed, offset, thresh, scale, drop_all, st);
    prof_mark(kProfAct, st, false);
    return err;
}

}  // namespace ms

// Device-side types and helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ms {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
// float -> bfloat16, round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }

// 16-byte vector of T (8 bf16 or 4 fp32).
template <typename T> struct Vec16 {
    static constexpr int N = 16 / sizeof(T);
    union {
        u32x4 u;
        T e[N];
    };
};

template <typename T>
__device__ __forceinline__ Vec16<T> load16(const T *p) {
    Vec16<T> v;
    v.u = *reinterpret_cast<const u32x4 *>(p);
    return v;
}

template <typename T>
__device__ __forceinline__ void store16(T *p, const Vec16<T> &v) {
    *reinterpret_cast<u32x4 *>(p) = v.u;
}

template <typename T>
__device__ __forceinline__ Vec16<T> zero16() {
    Vec16<T> v;
    v.u = u32x4{0u, 0u, 0u, 0u};
    return v;
}

// Eight consecutive elements of an elementwise pass (one 16-byte vector of
// bf16, two of fp32).  With VEC the whole group is read or written with
// 16-byte accesses when it lies inside [0, n) (the caller guarantees 16-byte
// alignment of the base); otherwise element by element, and elements past n
// read as zero and are not written.
template <typename T>
struct Group8 {
    T e[8];
};

template <typename T, bool VEC>
__device__ __forceinline__ Group8<T> load_group8(const T *__restrict__ p, int64_t i0, int64_t n) {
    Group8<T> g;
    if (VEC && i0 + 8 <= n) {
        const u32x4 *q = reinterpret_cast<const u32x4 *>(p + i0);
#pragma unroll
        for (int h = 0; h < (int)(8 * sizeof(T) / 16); ++h) reinterpret_cast<u32x4 *>(g.e)[h] = q[h];
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) g.e[e] = i0 + e < n ? p[i0 + e] : (T)0.f;
    }
    return g;
}

template <typename T, bool VEC>
__device__ __forceinline__ void store_group8(T *__restrict__ p, int64_t i0, int64_t n, const Group8<T> &g) {
    if (VEC && i0 + 8 <= n) {
        u32x4 *q = reinterpret_cast<u32x4 *>(p + i0);
#pragma unroll
        for (int h = 0; h < (int)(8 * sizeof(T) / 16); ++h) q[h] = reinterpret_cast<const u32x4 *>(g.e)[h];
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (i0 + e < n) p[i0 + e] = g.e[e];
    }
}

// Map a hardware block index to a logical tile index so that each of the 8
// XCDs (which receive blocks round-robin, block b -> XCD b % 8) owns one
// contiguous range of logical tiles: neighbouring tiles then share an L2.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
    const int X = 8;
    int q = nb / X, r = nb % X;
    int x = b % X, i = b / X;
    return (x < r) ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
}

}  // namespace ms

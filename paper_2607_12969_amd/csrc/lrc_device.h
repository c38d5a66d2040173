// Device-side building blocks for the gfx950 kernels: storage/accumulation
// types per precision, the 16x16 MFMA instructions used for each, fragment
// loads, wave reductions and the deterministic split-reduction handshake.
//
// MFMA convention used everywhere (16 x 16 output block, K step KB):
//   lane l supplies A-operand row (l & 15) and B-operand column (l & 15);
//   the K slice it supplies is [(l >> 4) * KPL, (l >> 4) * KPL + KPL) of the
//   step, the same slice for A and B, so the sum over K is exact whatever
//   order the hardware uses inside the step;
//   lane l receives D[row][l & 15] for v = 0..3 with row = acc_row<T>(l >> 4, v):
//   4 * (l >> 4) + v for the f32 and f16 instructions (four consecutive rows)
//   but (l >> 4) + 4 * v for v_mfma_f64_16x16x4_f64 (rows strided by 4).
// Kernels orient the MFMA so that the rows of D run along the output's
// contiguous dimension, so f32/f16 lanes hold four consecutive outputs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lrc {

typedef _Float16 half_t;
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));
typedef double double4_t __attribute__((ext_vector_type(4)));

template <typename T> struct PrecTraits;

// binary64 storage, binary64 accumulation: v_mfma_f64_16x16x4_f64
template <> struct PrecTraits<double> {
    using acc = double;
    using accv = double4_t;
    using frag = double;
    static constexpr int KPL = 1;   // K values per lane per MFMA
    static constexpr int KB = 4;    // K per MFMA
};

// binary32 storage, binary32 accumulation: v_mfma_f32_16x16x4_f32
template <> struct PrecTraits<float> {
    using acc = float;
    using accv = float4_t;
    using frag = float;
    static constexpr int KPL = 1;
    static constexpr int KB = 4;
};

// binary16 storage, binary32 accumulation: v_mfma_f32_16x16x32_f16 (gfx950)
template <> struct PrecTraits<half_t> {
    using acc = float;
    using accv = float4_t;
    using frag = half8_t;
    static constexpr int KPL = 8;
    static constexpr int KB = 32;
};

__device__ __forceinline__ double4_t mfma(double a, double b, double4_t c) {
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ float4_t mfma(float a, float b, float4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ float4_t mfma(half8_t a, half8_t b, float4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Row of the 16 x 16 MFMA result held in accumulator element v by lane
// group g = lane >> 4 (see the convention above).
template <typename T> __device__ __forceinline__ int acc_row(int g, int v) { return 4 * g + v; }
template <> __device__ __forceinline__ int acc_row<double>(int g, int v) { return g + 4 * v; }
// true when a lane's four accumulator rows are consecutive
template <typename T> struct AccRowsContiguous { static constexpr bool value = true; };
template <> struct AccRowsContiguous<double> { static constexpr bool value = false; };

template <typename T>
__device__ __forceinline__ typename PrecTraits<T>::frag load_frag(const T* p);

template <> __device__ __forceinline__ double load_frag<double>(const double* p) { return *p; }
template <> __device__ __forceinline__ float load_frag<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ half8_t load_frag<half_t>(const half_t* p) {
    return *reinterpret_cast<const half8_t*>(p);   // 16-byte aligned by construction
}

template <typename A>
__device__ __forceinline__ A zero_accv() {
    A z;
#pragma unroll
    for (int v = 0; v < 4; ++v) z[v] = 0;
    return z;
}

// Conversions from the accumulation type to the storage type use the
// hardware's round-to-nearest-even conversion (subnormals preserved).
template <typename T, typename Acc>
__device__ __forceinline__ T to_storage(Acc x) { return static_cast<T>(x); }

template <typename T>
__device__ __forceinline__ typename PrecTraits<T>::acc to_acc(T x) {
    return static_cast<typename PrecTraits<T>::acc>(x);
}

// Sum over the 64 lanes of a wavefront, fixed butterfly order.
template <typename Acc>
__device__ __forceinline__ Acc wave_sum(Acc x) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
    return x;
}

// Workgroups are handed to the 8 XCDs in turn (workgroup L to XCD L mod 8).
// Renumber them so that XCD x works through the contiguous range
// [x R, (x + 1) R) of logical tiles, R = ceil(total / 8), whose shared
// operands then meet in that XCD's L2.  The grid is padded to 8 R
// workgroups (xcd_grid); the numbers past `total` belong to no tile.
__device__ __forceinline__ int64_t xcd_tile(int64_t total) {
    const int64_t L = blockIdx.x;
    return (L % 8) * ((total + 7) / 8) + L / 8;
}
static inline unsigned xcd_grid(int64_t total) { return (unsigned)(((total + 7) / 8) * 8); }

}  // namespace lrc

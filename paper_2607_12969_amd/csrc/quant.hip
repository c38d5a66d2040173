// Device quantization: binary64 values rounded to the storage formats.
//
// The stored representation of the method is every factor (or TT core)
// entry rounded on its own from binary64 to binary32 or binary16 (Sec. 3.2
// formats; the Remark after Thm thm:matrix_rank_compensation; Algorithm
// alg:tt_compensation, rounding step).  Each value takes ONE
// round-to-nearest-even step; binary16 subnormals are kept.
//
// k_round is an HBM-bound stream: 8 bytes read and e bytes written per
// value, four values per lane and step (two 16-byte loads, one 8- or
// 16-byte store) when the pointers allow it.
#include <hip/hip_runtime.h>

#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

// binary64 -> binary16, one rounding step, ties to even, from the bit
// fields.  A binary64 value is S 2^(E-52) with the 53-bit significand S;
// the binary16 quantum at exponent E is 2^(max(E, -14) - 10), so S loses
// `sh` = 42 + max(0, -14 - E) low bits.  The kept part q, rounded, is the
// encoding itself up to the exponent field: normals ((E + 14) << 10) + q
// with q in [2^10, 2^11] (a carry to 2^11 moves into the exponent),
// subnormals q in [0, 2^10] (2^10 is the smallest normal, 0x0400).
// Encodings from 0x7C00 up are overflows to infinity.  NaN gives the quiet
// NaN of the same sign; binary64 subnormals (below 2^-1022) give zero.
__device__ __forceinline__ uint16_t f64_to_f16_bits(double v, int& overflow) {
    const uint64_t b = (uint64_t)__double_as_longlong(v);
    const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
    const int e = (int)((b >> 52) & 0x7FF);
    const uint64_t frac = b & 0xFFFFFFFFFFFFFull;
    if (e == 0x7FF) return (uint16_t)(sign | (frac ? 0x7E00u : 0x7C00u));
    if (e == 0) return sign;
    const int E = e - 1023;
    const int sh = 42 + (E < -14 ? -14 - E : 0);
    // S < 2^53, so for sh >= 54 the value is below half the smallest
    // subnormal (a tie there is impossible): it rounds to zero
    if (sh >= 54) return sign;
    const uint64_t S = frac | (1ull << 52);
    uint64_t q = S >> sh;
    const uint64_t rem = S & ((1ull << sh) - 1), half = 1ull << (sh - 1);
    q += (rem > half || (rem == half && (q & 1))) ? 1 : 0;
    const int64_t enc = E >= -14 ? ((int64_t)(E + 14) << 10) + (int64_t)q : (int64_t)q;
    if (enc >= 0x7C00) {
        overflow += 1;
        return (uint16_t)(sign | 0x7C00u);
    }
    return (uint16_t)(sign | (uint16_t)enc);
}

// binary64 -> binary32: the hardware conversion rounds to nearest even
// (the default mode) and keeps binary32 subnormals; NaN is mapped to the
// quiet NaN of the same sign so the bits do not depend on the payload.
__device__ __forceinline__ uint32_t f64_to_f32_bits(double v, int& overflow) {
    if (v != v) return (__double_as_longlong(v) < 0 ? 0x80000000u : 0u) | 0x7FC00000u;
    const float f = (float)v;
    const uint32_t u = __float_as_uint(f);
    if ((u & 0x7FFFFFFFu) == 0x7F800000u && __builtin_fabs(v) <= 1.7976931348623157e308) overflow += 1;
    return u;
}

template <typename U>
__device__ __forceinline__ U round_bits(double v, int& overflow);
template <> __device__ __forceinline__ uint16_t round_bits<uint16_t>(double v, int& overflow) {
    return f64_to_f16_bits(v, overflow);
}
template <> __device__ __forceinline__ uint32_t round_bits<uint32_t>(double v, int& overflow) {
    return f64_to_f32_bits(v, overflow);
}

// y[i] = round(x[i]) for i < n, as storage bits U (uint16_t / uint32_t).
// VEC: x 16-byte and y (4 sizeof(U))-byte aligned; every lane then takes
// four consecutive values per step.  Finite inputs that overflow are
// counted into *ovf (integer atomics: the count does not depend on order)
// when ovf is not null.
template <typename U, bool VEC>
__global__ __launch_bounds__(256) void k_round(const double* __restrict__ x, U* __restrict__ y, int64_t n,
                                               unsigned long long* __restrict__ ovf) {
    int over = 0;
    const int64_t stride = (int64_t)gridDim.x * 256;
    const int64_t t0 = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (VEC) {
        typedef double d2_t __attribute__((ext_vector_type(2)));
        typedef U u4_t __attribute__((ext_vector_type(4)));
        const int64_t n4 = n / 4;
        for (int64_t q = t0; q < n4; q += stride) {
            const d2_t a = __builtin_nontemporal_load(reinterpret_cast<const d2_t*>(x) + 2 * q);
            const d2_t b = __builtin_nontemporal_load(reinterpret_cast<const d2_t*>(x) + 2 * q + 1);
            u4_t w;
            w[0] = round_bits<U>(a[0], over);
            w[1] = round_bits<U>(a[1], over);
            w[2] = round_bits<U>(b[0], over);
            w[3] = round_bits<U>(b[1], over);
            __builtin_nontemporal_store(w, reinterpret_cast<u4_t*>(y) + q);
        }
        for (int64_t i = 4 * n4 + t0; i < n; i += stride) y[i] = round_bits<U>(x[i], over);
    } else {
        for (int64_t i = t0; i < n; i += stride) y[i] = round_bits<U>(x[i], over);
    }
    if (ovf) {
        // one atomic per wave
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) over += __shfl_xor(over, off, 64);
        if ((threadIdx.x & 63) == 0 && over) atomicAdd(ovf, (unsigned long long)over);
    }
}

__global__ void k_zero_u64(unsigned long long* p) { *p = 0ull; }

hipError_t launch_round(const double* x, void* y, int64_t n, int prec, unsigned long long* ovf,
                        hipStream_t stream) {
    if (ovf) hipLaunchKernelGGL(k_zero_u64, dim3(1), dim3(1), 0, stream, ovf);
    if (n == 0) return hipGetLastError();
    KernelTimer t("quant_round", stream);
    // enough waves to keep HBM busy; each lane handles 4 values per step
    int64_t g = (n / 4 + 255) / 256;
    if (g > 8192) g = 8192;
    if (g < 1) g = 1;
    const bool xa = reinterpret_cast<uintptr_t>(x) % 16 == 0;
    if (prec == P32) {
        const bool vec = xa && reinterpret_cast<uintptr_t>(y) % 16 == 0;
        if (vec)
            hipLaunchKernelGGL((k_round<uint32_t, true>), dim3(g), dim3(256), 0, stream, x, (uint32_t*)y, n, ovf);
        else
            hipLaunchKernelGGL((k_round<uint32_t, false>), dim3(g), dim3(256), 0, stream, x, (uint32_t*)y, n, ovf);
    } else {
        const bool vec = xa && reinterpret_cast<uintptr_t>(y) % 8 == 0;
        if (vec)
            hipLaunchKernelGGL((k_round<uint16_t, true>), dim3(g), dim3(256), 0, stream, x, (uint16_t*)y, n, ovf);
        else
            hipLaunchKernelGGL((k_round<uint16_t, false>), dim3(g), dim3(256), 0, stream, x, (uint16_t*)y, n, ovf);
    }
    return hipGetLastError();
}

}  // namespace lrc

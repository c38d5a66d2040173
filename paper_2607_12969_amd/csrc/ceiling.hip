// Matrix-core ceiling of this device, for the roofline fractions reported
// against measured peaks next to the published ones: every wave runs a loop
// of eight independent MFMAs of the instruction the kernels use (FP64
// 16x16x4, FP32 16x16x4, FP16 16x16x32 with FP32 accumulation) on operands
// held in registers, so nothing but the matrix unit is timed.  The sums are
// written out so that the loop is not removed.
#include <hip/hip_runtime.h>

#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

constexpr int kCeilWaves = 4;          // per workgroup
constexpr int kCeilGroupsPerCU = 8;    // workgroups per compute unit

template <typename T>
__global__ __launch_bounds__(64 * kCeilWaves) void k_mfma_ceiling(int iters, typename PrecTraits<T>::accv* out) {
    using Frag = typename PrecTraits<T>::frag;
    using AccV = typename PrecTraits<T>::accv;
    const int lane = threadIdx.x & 63;
    Frag a, b;
    if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            a[j] = (half_t)(0.001f * (float)((lane + j) & 7));
            b[j] = (half_t)(0.002f * (float)((lane * 3 + j) & 7));
        }
    } else {
        a = (T)(0.001 * (lane & 7));
        b = (T)(0.002 * ((lane * 3) & 7));
    }
    AccV acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = zero_accv<AccV>();
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] = mfma(a, b, acc[j]);
    }
    AccV s = acc[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) s += acc[j];
    out[(int64_t)blockIdx.x * (64 * kCeilWaves) + threadIdx.x] = s;
}

// flops of one MFMA of the kernels' instruction
template <typename T> constexpr double mfma_flops() { return sizeof(T) == 2 ? 16.0 * 16 * 32 * 2 : 16.0 * 16 * 4 * 2; }

template <typename T>
static hipError_t ceiling_typed(int cus, double seconds_target, double* tflops, Workspace& ws, hipStream_t st) {
    using AccV = typename PrecTraits<T>::accv;
    const int groups = cus * kCeilGroupsPerCU;
    AccV* out = static_cast<AccV*>(ws.take((size_t)groups * 64 * kCeilWaves * sizeof(AccV)));
    if (ws.overrun || !out) return hipErrorOutOfMemory;
    const double peak = sizeof(T) == 8 ? 78.6e12 : (sizeof(T) == 4 ? 157.3e12 : 2500e12);
    const double per_iter = mfma_flops<T>() * 8.0 * kCeilWaves * groups;
    const int iters = (int)std::max(64.0, std::min(1e6, seconds_target * peak / per_iter));
    hipEvent_t e0, e1;
    hipError_t e = hipEventCreate(&e0);
    if (e != hipSuccess) return e;
    e = hipEventCreate(&e1);
    if (e != hipSuccess) {
        hipEventDestroy(e0);
        return e;
    }
    float best = 0.0f;
    for (int rep = 0; rep < 3 && e == hipSuccess; ++rep) {   // the first run warms the clocks
        e = hipEventRecord(e0, st);
        if (e == hipSuccess) {
            hipLaunchKernelGGL(k_mfma_ceiling<T>, dim3(groups), dim3(64 * kCeilWaves), 0, st, iters, out);
            e = hipGetLastError();
        }
        if (e == hipSuccess) e = hipEventRecord(e1, st);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float ms = 0.0f;
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
        if (e == hipSuccess && rep > 0 && (best == 0.0f || ms < best)) best = ms;
    }
    hipEventDestroy(e0);
    hipEventDestroy(e1);
    if (e != hipSuccess) return e;
    *tflops = per_iter * iters / (best * 1e-3) / 1e12;
    return hipSuccess;
}

size_t mfma_ceiling_workspace_bytes(int cus) {
    return (size_t)cus * kCeilGroupsPerCU * 64 * kCeilWaves * 4 * sizeof(double) + 256;
}

hipError_t launch_mfma_ceiling(int prec, int cus, double* tflops, Workspace& ws, hipStream_t st) {
    if (prec == P64) return ceiling_typed<double>(cus, 0.01, tflops, ws, st);
    if (prec == P32) return ceiling_typed<float>(cus, 0.01, tflops, ws, st);
    return ceiling_typed<half_t>(cus, 0.01, tflops, ws, st);
}

}  // namespace lrc

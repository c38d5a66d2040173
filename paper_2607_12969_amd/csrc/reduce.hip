// Element-wise preparation and deterministic reductions for the device-side
// certificate (Thm thm:matrix_rank_compensation, Thm thm:tt_conditional).
//
// Every reduction here has a fixed shape: a grid of a fixed number of
// workgroups, each thread summing a fixed strided subset in ascending order,
// a fixed butterfly inside the wavefront and wave order inside the
// workgroup, then one workgroup summing the per-workgroup partials in index
// order.  Results are therefore bitwise reproducible and never use
// floating-point atomics.
#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

template <typename T>
__device__ __forceinline__ double widen1(T x) { return static_cast<double>(x); }

// P[i][t] = ref[i][t];  P[i][r + t] = widen(h[i][t]) - ref[i][t]
// The difference of a value and its rounding is exact in binary64, so the
// second block holds the rounding perturbation itself.
template <typename T>
__global__ __launch_bounds__(256) void k_diff_factors(const double* __restrict__ ref, const T* __restrict__ h,
                                                      int64_t rows, int64_t r, double* __restrict__ P) {
    const int64_t total = rows * r;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total; idx += (int64_t)gridDim.x * 256) {
        const int64_t i = idx / r, t = idx % r;
        const double a = ref[idx];
        P[i * 2 * r + t] = a;
        P[i * 2 * r + r + t] = widen1(h[idx]) - a;
    }
}

// W[i][t] = widen(h[i][t]) * widen(hs[t]); the product of two stored values
// is exact in binary64 (at most 2 x 24 significand bits).
template <typename T>
__global__ __launch_bounds__(256) void k_widen_scaled(const T* __restrict__ h, const T* __restrict__ hs,
                                                      int64_t rows, int64_t r, int64_t ldw,
                                                      double* __restrict__ W) {
    const int64_t total = rows * ldw;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total; idx += (int64_t)gridDim.x * 256) {
        const int64_t i = idx / ldw, t = idx % ldw;
        double v = 0.0;
        if (t < r) v = widen1(h[i * r + t]) * (hs ? widen1(hs[t]) : 1.0);
        W[idx] = v;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void k_widen(const T* __restrict__ src, int64_t count, double* __restrict__ out) {
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < count; idx += (int64_t)gridDim.x * 256)
        out[idx] = widen1(src[idx]);
}

static unsigned grid_for(int64_t total) {
    int64_t g = (total + 255) / 256;
    if (g > 4096) g = 4096;
    if (g < 1) g = 1;
    return (unsigned)g;
}

hipError_t launch_diff_factors(const double* ref, const void* h, int prec, int64_t rows, int64_t r, double* P,
                               hipStream_t stream) {
    const unsigned g = grid_for(rows * r);
    KernelTimer tm("cert_diff_factors", stream);
    if (prec == P64)
        hipLaunchKernelGGL(k_diff_factors<double>, dim3(g), dim3(256), 0, stream, ref, (const double*)h, rows, r, P);
    else if (prec == P32)
        hipLaunchKernelGGL(k_diff_factors<float>, dim3(g), dim3(256), 0, stream, ref, (const float*)h, rows, r, P);
    else
        hipLaunchKernelGGL(k_diff_factors<half_t>, dim3(g), dim3(256), 0, stream, ref, (const half_t*)h, rows, r, P);
    return hipGetLastError();
}

hipError_t launch_widen_scaled(const void* h, const void* hs, int prec, int64_t rows, int64_t r, int64_t ldw,
                               double* W, hipStream_t stream) {
    const unsigned g = grid_for(rows * ldw);
    KernelTimer tm("cert_widen", stream);
    if (prec == P64)
        hipLaunchKernelGGL(k_widen_scaled<double>, dim3(g), dim3(256), 0, stream, (const double*)h, (const double*)hs, rows, r, ldw, W);
    else if (prec == P32)
        hipLaunchKernelGGL(k_widen_scaled<float>, dim3(g), dim3(256), 0, stream, (const float*)h, (const float*)hs, rows, r, ldw, W);
    else
        hipLaunchKernelGGL(k_widen_scaled<half_t>, dim3(g), dim3(256), 0, stream, (const half_t*)h, (const half_t*)hs, rows, r, ldw, W);
    return hipGetLastError();
}

hipError_t launch_widen(const void* src, int prec, int64_t count, double* out, hipStream_t stream) {
    const unsigned g = grid_for(count);
    KernelTimer tm("cert_widen", stream);
    if (prec == P64)
        hipLaunchKernelGGL(k_widen<double>, dim3(g), dim3(256), 0, stream, (const double*)src, count, out);
    else if (prec == P32)
        hipLaunchKernelGGL(k_widen<float>, dim3(g), dim3(256), 0, stream, (const float*)src, count, out);
    else
        hipLaunchKernelGGL(k_widen<half_t>, dim3(g), dim3(256), 0, stream, (const half_t*)src, count, out);
    return hipGetLastError();
}

// Five sums over a dense tensor of `count` entries:
//   q=0 (T-a)^2   q=1 (T-b)^2   q=2 (b-c)^2   q=3 (T-c)^2   q=4 T^2
// with a = T_R, b = T_{R+}, c = the tensor of the rounded cores.
__global__ __launch_bounds__(256) void k_sumsq5(const double* __restrict__ T, const double* __restrict__ a,
                                                const double* __restrict__ b, const double* __restrict__ c,
                                                int64_t count, double* __restrict__ part) {
    __shared__ double red[5][4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    double s[5] = {0.0, 0.0, 0.0, 0.0, 0.0};
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + tid; i < count; i += stride) {
        const double t = T[i], x = a[i], y = b[i], z = c[i];
        const double d0 = t - x, d1 = t - y, d2 = y - z, d3 = t - z;
        s[0] += d0 * d0;
        s[1] += d1 * d1;
        s[2] += d2 * d2;
        s[3] += d3 * d3;
        s[4] += t * t;
    }
#pragma unroll
    for (int q = 0; q < 5; ++q) {
        const double w = wave_sum(s[q]);
        if (lane == 0) red[q][wave] = w;
    }
    __syncthreads();
    if (tid < 5) {
        const double t = ((red[tid][0] + red[tid][1]) + red[tid][2]) + red[tid][3];
        part[(int64_t)tid * gridDim.x + blockIdx.x] = t;
    }
}

int64_t sumsq5_groups(int64_t count) {
    int64_t g = (count + 255) / 256;
    if (g > 1024) g = 1024;
    if (g < 1) g = 1;
    return g;
}

hipError_t launch_sumsq5(const double* T, const double* a, const double* b, const double* c, int64_t count,
                         double* part, int64_t groups, hipStream_t stream) {
    KernelTimer tm("cert_sumsq5_f64", stream);
    hipLaunchKernelGGL(k_sumsq5, dim3((unsigned)groups), dim3(256), 0, stream, T, a, b, c, count, part);
    return hipGetLastError();
}

// eta^2 = ||P M Q^T||_F^2 = trace(M^T Gu M Gq) for the matrix certificate
// (Thm. thm:matrix_rank_compensation), with P = [U dU], Q = [V dV] and
//   M = [[dS, S^], [S^, S^]]  (rows U | dU, columns V | dV),
// since A^_{k+1} - A_{k+1} = U dS V^T + U S^ dV^T + dU S^ V^T + dU S^ dV^T.
// Every term has the size of the perturbation, so nothing of the size of
// ||A|| cancels.  Column a of M has two non-zeros:
//   a < r : M[a][a] = dS_a,      M[r+a][a] = S^_a
//   a >= r: M[a-r][a] = S^_{a-r}, M[a][a]  = S^_{a-r}
// Workgroup ca writes part[ca] = sum_cb (M^T Gu M)[ca][cb] * Gq[cb][ca],
// each term summed in a fixed order.
// shv = S^ of the column's index modulo r
__device__ __forceinline__ void eta_nz(int64_t col, int64_t r, const double* s, double shv, int64_t* rows,
                                       double* vals) {
    if (col < r) {
        rows[0] = col;
        vals[0] = shv - s[col];
        rows[1] = r + col;
        vals[1] = shv;
    } else {
        rows[0] = col - r;
        vals[0] = shv;
        rows[1] = col;
        vals[1] = shv;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void k_eta2(const double* __restrict__ Gu, const double* __restrict__ Gq,
                                              const double* __restrict__ s, const T* __restrict__ sh, int64_t r,
                                              double* __restrict__ part) {
    __shared__ double red[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t w2 = 2 * r;
    const int64_t ca = blockIdx.x;
    int64_t ra[2];
    double va[2];
    eta_nz(ca, r, s, widen1(sh[ca < r ? ca : ca - r]), ra, va);
    double acc = 0.0;
    for (int64_t cb = tid; cb < w2; cb += 256) {
        int64_t rb[2];
        double vb[2];
        eta_nz(cb, r, s, widen1(sh[cb < r ? cb : cb - r]), rb, vb);
        double h = 0.0;
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) h += va[x] * Gu[ra[x] * w2 + rb[y]] * vb[y];
        acc += h * Gq[cb * w2 + ca];
    }
    acc = wave_sum(acc);
    if (lane == 0) red[wave] = acc;
    __syncthreads();
    if (tid == 0) part[ca] = ((red[0] + red[1]) + red[2]) + red[3];
}

hipError_t launch_eta2(const double* Gu, const double* Gq, const double* s, const void* sh, int prec, int64_t r,
                       double* part, hipStream_t stream) {
    KernelTimer tm("cert_eta2_f64", stream);
    const dim3 g((unsigned)(2 * r));
    if (prec == P64)
        hipLaunchKernelGGL(k_eta2<double>, g, dim3(256), 0, stream, Gu, Gq, s, (const double*)sh, r, part);
    else if (prec == P32)
        hipLaunchKernelGGL(k_eta2<float>, g, dim3(256), 0, stream, Gu, Gq, s, (const float*)sh, r, part);
    else
        hipLaunchKernelGGL(k_eta2<half_t>, g, dim3(256), 0, stream, Gu, Gq, s, (const half_t*)sh, r, part);
    return hipGetLastError();
}

// One workgroup per row: out[row] = sum_j part[row][j], fixed order.
__global__ __launch_bounds__(256) void k_reduce_rows(const double* __restrict__ part, int64_t count,
                                                     double* __restrict__ out) {
    __shared__ double red[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const double* p = part + (int64_t)blockIdx.x * count;
    double s = 0.0;
    for (int64_t j = tid; j < count; j += 256) s += p[j];
    s = wave_sum(s);
    if (lane == 0) red[wave] = s;
    __syncthreads();
    if (tid == 0) out[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

hipError_t launch_reduce_rows(const double* part, int64_t count, int nsums, double* out, hipStream_t stream) {
    KernelTimer tm("cert_reduce_rows", stream);
    hipLaunchKernelGGL(k_reduce_rows, dim3(nsums), dim3(256), 0, stream, part, count, out);
    return hipGetLastError();
}

}  // namespace lrc

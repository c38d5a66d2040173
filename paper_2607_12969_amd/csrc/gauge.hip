// Left-orthogonal gauge of an FP64 Tensor Train (Sec. 6.1; Algorithm
// alg:tt_compensation, gauge step): for l = 1..d-1 the left unfolding of
// core l, A = G_l as (r_{l-1} n_l) x r_l, is factored A = Q R with
// Q^T Q = I and diag(R) > 0; core l becomes Q and R is multiplied into the
// left unfolding of core l+1 (r_l x n_{l+1} r_{l+1}).
//
// The QR of each unfolding is CholeskyQR2: with the Gram matrix A^T A = R_1^T
// R_1 (Cholesky), Q_1 = A R_1^{-1}; then Q_1^T Q_1 = R_2^T R_2, Q = Q_1
// R_2^{-1} and R = R_2 R_1.  The first pass leaves an orthogonality error of
// order cond(A)^2 u, the second removes it while cond(A)^2 u stays well
// below one; the Cholesky stops with an error when a pivot falls below 2^-46
// of its column's squared norm (cond(A) above about 10^7), where the
// factorization would no longer be accurate.  With positive diagonals both
// R and Q are the unique thin QR factors of a full-rank A, so the result
// agrees to rounding with a Householder QR of the same convention.
//
// Work per unfolding (m rows, r columns): two Gram products on the FP64
// matrix cores (launch_gram: 2 m r^2 flop each, half of it computed), two
// row products with a triangular r x r matrix (m r^2 flop each), and the
// product R G_{l+1} (2 r^2 n_{l+1} r_{l+1} flop).  All of it is small next
// to the reconstruction; the kernels are plain FP64 vector code except the
// Gram.
#include <hip/hip_runtime.h>

#include "../../include/lrc.h"
#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

// dst[i][j] = src[i][j] for j < r, 0 for r <= j < ldd (rows x ldd)
__global__ __launch_bounds__(256) void k_gauge_pad(const double* __restrict__ src, int64_t rows, int r,
                                                   double* __restrict__ dst, int ldd) {
    const int64_t total = rows * ldd;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total; idx += (int64_t)gridDim.x * 256) {
        const int64_t i = idx / ldd;
        const int j = (int)(idx - i * ldd);
        dst[idx] = j < r ? src[i * r + j] : 0.0;
    }
}

// One workgroup.  G (r x r inside pitch ld, symmetric, upper triangle used)
// = R^T R with R upper triangular, diag(R) > 0 (right-looking Cholesky in
// LDS).  Writes R and its inverse Rinv (both upper, zero below the diagonal
// and in the pad columns up to ld) and, when Rprev is given, Rout = R Rprev.
// flag: set to 1 + (pivot index) when a pivot is not above 2^-46 of the
// column's original diagonal (or not a number); the outputs are then
// unspecified.
constexpr int kGaugeMaxRank = LRC_GAUGE_MAX_RANK;
__global__ __launch_bounds__(256) void k_gauge_chol(const double* __restrict__ G, int r, int ld,
                                                    double* __restrict__ R, double* __restrict__ Rinv,
                                                    const double* __restrict__ Rprev, double* __restrict__ Rout,
                                                    int* __restrict__ flag) {
    __shared__ double S[kGaugeMaxRank][kGaugeMaxRank + 1];
    __shared__ double diag0[kGaugeMaxRank];
    __shared__ int bad;
    const int tid = threadIdx.x;
    for (int idx = tid; idx < r * r; idx += 256) {
        const int i = idx / r, j = idx - i * r;
        S[i][j] = j >= i ? G[(int64_t)i * ld + j] : 0.0;
    }
    if (tid == 0) bad = 0;
    __syncthreads();
    for (int i = tid; i < r; i += 256) diag0[i] = S[i][i];
    __syncthreads();
    for (int k = 0; k < r; ++k) {
        if (tid == 0) {
            const double d = S[k][k];
            // a pivot that is not positive relative to its column (NaN fails too)
            if (!(d > 0x1p-46 * diag0[k]) && bad == 0) bad = 1 + k;
            S[k][k] = __builtin_sqrt(d > 0.0 ? d : 0.0);
        }
        __syncthreads();
        const double rkk = S[k][k];
        for (int j = k + 1 + tid; j < r; j += 256) S[k][j] = S[k][j] / rkk;
        __syncthreads();
        // trailing update of the upper triangle: S[i][j] -= R[k][i] R[k][j], k < i <= j
        const int t = r - k - 1;
        for (int idx = tid; idx < t * t; idx += 256) {
            const int i = k + 1 + idx / t, j = k + 1 + idx % t;
            if (j >= i) S[i][j] -= S[k][i] * S[k][j];
        }
        __syncthreads();
    }
    if (tid == 0 && bad) *flag = bad;
    for (int idx = tid; idx < r * ld; idx += 256) {
        const int i = idx / ld, j = idx - i * ld;
        R[(int64_t)i * ld + j] = (j < r && j >= i) ? S[i][j] : 0.0;
    }
    // Rinv column j by back substitution (thread j); entries below the
    // diagonal and in the pad are zero
    for (int j = tid; j < ld; j += 256) {
        for (int i = ld - 1; i >= 0; --i) {
            double v = 0.0;
            if (j < r && i <= j) {
                double acc = (i == j) ? 1.0 : 0.0;
                for (int q = i + 1; q <= j; ++q) acc -= S[i][q] * Rinv[(int64_t)q * ld + j];
                v = acc / S[i][i];
            }
            Rinv[(int64_t)i * ld + j] = v;
        }
    }
    if (Rprev) {
        __syncthreads();
        // Rout = R Rprev, both upper triangular
        for (int idx = tid; idx < r * ld; idx += 256) {
            const int i = idx / ld, j = idx - i * ld;
            double acc = 0.0;
            if (j < r && j >= i)
                for (int q = i; q <= j; ++q) acc += S[i][q] * Rprev[(int64_t)q * ld + j];
            Rout[(int64_t)i * ld + j] = acc;
        }
    }
}

// C[i][j] = sum_{t <= j} A[i][t] B[t][j] for j < r (B upper triangular,
// pitch ldb); C has pitch ldc, and pad columns r <= j < ldc are zeroed.
// One wave per row, lane j (and j + 64) per output column; lane t holds
// A[i][t] (and A[i][t + 64]) and hands it to the wave by a lane shuffle, so
// B's rows are read coalesced and A once.
__global__ __launch_bounds__(256) void k_gauge_rmul(const double* __restrict__ A, int64_t rows, int r, int lda,
                                                    const double* __restrict__ B, int ldb,
                                                    double* __restrict__ C, int ldc) {
    const int lane = threadIdx.x & 63;
    const int64_t w0 = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t ws = (int64_t)gridDim.x * 4;
    for (int64_t i = w0; i < rows; i += ws) {
        const double* a = A + i * lda;
        const double a0 = lane < r ? a[lane] : 0.0;
        const double a1 = lane + 64 < r ? a[lane + 64] : 0.0;
        double c0 = 0.0, c1 = 0.0;
        for (int t = 0; t < r; ++t) {
            const double at = t < 64 ? __shfl(a0, t, 64) : __shfl(a1, t - 64, 64);
            const double* b = B + (int64_t)t * ldb;
            if (lane < r && t <= lane) c0 += at * b[lane];
            if (lane + 64 < r && t <= lane + 64) c1 += at * b[lane + 64];
        }
        double* c = C + i * ldc;
        if (lane < ldc) c[lane] = lane < r ? c0 : 0.0;
        if (lane + 64 < ldc) c[lane + 64] = lane + 64 < r ? c1 : 0.0;
    }
}

// C[i][c] = sum_{t >= i} R[i][t] X[t][c] for i < r, c < ncols (R upper
// triangular with pitch ldr, X and C r x ncols dense).  One thread per
// column c: the column of X is read once (coalesced across threads) into
// registers in chunks of 32 rows, and R is read at uniform addresses.
__global__ __launch_bounds__(256) void k_gauge_lmul(const double* __restrict__ R, int r, int ldr,
                                                    const double* __restrict__ X, int64_t ncols,
                                                    double* __restrict__ C) {
    const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (c >= ncols) return;
    for (int i0 = 0; i0 < r; i0 += 32) {
        double acc[32];
#pragma unroll
        for (int u = 0; u < 32; ++u) acc[u] = 0.0;
        // rows t >= i0 contribute to outputs i0 .. i0 + 31
        for (int t = i0; t < r; ++t) {
            const double x = X[(int64_t)t * ncols + c];
            const double* rt = R + t;   // R[i][t] = rt[i * ldr]
#pragma unroll
            for (int u = 0; u < 32; ++u) {
                const int i = i0 + u;
                if (i < r && i <= t) acc[u] += rt[(int64_t)i * ldr] * x;
            }
        }
#pragma unroll
        for (int u = 0; u < 32; ++u)
            if (i0 + u < r) C[(int64_t)(i0 + u) * ncols + c] = acc[u];
    }
}

static unsigned gauge_grid(int64_t items, int per_block) {
    int64_t g = (items + per_block - 1) / per_block;
    if (g > 8192) g = 8192;
    return (unsigned)(g < 1 ? 1 : g);
}

size_t gauge_workspace_bytes(const int64_t* dims, const int64_t* ranks, int d) {
    size_t need = 0;
    for (int l = 0; l + 1 < d; ++l) {
        const int64_t rows = ranks[l] * dims[l], r = ranks[l + 1];
        const int64_t rp = round_up(r, 2);
        const int64_t ncols = dims[l + 1] * ranks[l + 2];
        size_t b = 0;
        b += round_up((int64_t)(rows * rp * 8), 256) * 2;                   // W1, W2
        b += round_up((int64_t)(rp * rp * 8), 256) * 6;                     // G, R1, Rinv1, R2, Rinv2, R
        b += round_up((int64_t)gram_workspace_bytes(rows, rp), 256);        // Gram partials
        b += round_up((int64_t)(r * ncols * 8), 256);                       // R G_{l+1}
        need = b > need ? b : need;
    }
    return need + 256 + (size_t)round_up(4 * (int64_t)d, 256);
}

__global__ void k_gauge_zero(int* p, int n) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

hipError_t launch_gauge(double* const* cores, const int64_t* dims, const int64_t* ranks, int d, int* flags,
                        Workspace& ws, hipStream_t stream) {
    hipLaunchKernelGGL(k_gauge_zero, dim3(1), dim3(64), 0, stream, flags, d);
    for (int l = 0; l + 1 < d; ++l) {
        const int64_t rows = ranks[l] * dims[l];
        const int r = (int)ranks[l + 1];
        const int rp = (int)round_up(r, 2);
        const int64_t ncols = dims[l + 1] * ranks[l + 2];
        const size_t mark = ws.used;
        double* W1 = static_cast<double*>(ws.take((size_t)rows * rp * 8));
        double* W2 = static_cast<double*>(ws.take((size_t)rows * rp * 8));
        double* G = static_cast<double*>(ws.take((size_t)rp * rp * 8));
        double* R1 = static_cast<double*>(ws.take((size_t)rp * rp * 8));
        double* I1 = static_cast<double*>(ws.take((size_t)rp * rp * 8));
        double* R2 = static_cast<double*>(ws.take((size_t)rp * rp * 8));
        double* I2 = static_cast<double*>(ws.take((size_t)rp * rp * 8));
        double* Rt = static_cast<double*>(ws.take((size_t)rp * rp * 8));
        double* NX = static_cast<double*>(ws.take((size_t)r * ncols * 8));
        if (ws.overrun) return hipErrorOutOfMemory;
        KernelTimer tm("gauge_qr_f64", stream);
        hipLaunchKernelGGL(k_gauge_pad, dim3(gauge_grid(rows * rp, 256)), dim3(256), 0, stream, cores[l], rows, r,
                           W1, rp);
        // first pass: A^T A = R1^T R1, W2 = A R1^{-1}
        const size_t gmark = ws.used;
        hipError_t e = launch_gram(W1, rows, rp, G, ws, stream);
        if (e != hipSuccess) return e;
        ws.used = gmark;
        hipLaunchKernelGGL(k_gauge_chol, dim3(1), dim3(256), 0, stream, G, r, rp, R1, I1, (const double*)nullptr,
                           (double*)nullptr, flags + l);
        hipLaunchKernelGGL(k_gauge_rmul, dim3(gauge_grid(rows, 4)), dim3(256), 0, stream, W1, rows, r, rp, I1, rp,
                           W2, rp);
        // second pass on W2: R = R2 R1, core l = W2 R2^{-1}
        e = launch_gram(W2, rows, rp, G, ws, stream);
        if (e != hipSuccess) return e;
        ws.used = gmark;
        hipLaunchKernelGGL(k_gauge_chol, dim3(1), dim3(256), 0, stream, G, r, rp, R2, I2, R1, Rt, flags + l);
        hipLaunchKernelGGL(k_gauge_rmul, dim3(gauge_grid(rows, 4)), dim3(256), 0, stream, W2, rows, r, rp, I2, rp,
                           cores[l], r);
        // core l+1 <- R core l+1 (left unfolding r x ncols)
        hipLaunchKernelGGL(k_gauge_lmul, dim3(gauge_grid(ncols, 256)), dim3(256), 0, stream, Rt, r, rp,
                           cores[l + 1], ncols, NX);
        e = hipMemcpyAsync(cores[l + 1], NX, (size_t)r * ncols * 8, hipMemcpyDeviceToDevice, stream);
        if (e != hipSuccess) return e;
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        ws.used = mark;
    }
    return hipSuccess;
}

}  // namespace lrc

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
// triangular solves x R = a per row (forward substitution, m r^2 flop
// each; no inverse is formed), and R G_{l+1} applied as R_2 (R_1 G_{l+1})
// (two triangular products, r^2 n_{l+1} r_{l+1} flop each).  All of it is
// small next to the reconstruction; the kernels are plain FP64 vector code
// except the Gram.
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
// = R^T R with R upper triangular, diag(R) > 0: right-looking Cholesky in
// LDS with one barrier per pivot (the trailing update uses the unscaled
// pivot row, S[i][j] -= S[k][i] S[k][j] / S[k][k], while row k of R goes to
// a matrix of its own).  R is written with pitch ld, zero below the diagonal and in
// the pad rows and columns.  flag: set to 1 + (pivot index) when a pivot is
// not above 2^-46 of the column's original diagonal (or not a number); R is
// then unspecified.  shift_rel > 0 factors G + s I instead, s = shift_rel
// trace(G) (the shifted first pass of shifted CholeskyQR3).
constexpr int kGaugeMaxRank = LRC_GAUGE_MAX_RANK;
constexpr int kCholSide = 32;                          // the Cholesky's thread grid is kCholSide^2
constexpr int kCholThreads = kCholSide * kCholSide;

// S[i][j] = M[i][j] (pitch ld) for j >= i, 0 below the diagonal, i, j < r,
// by NTH threads: every thread issues all its global loads before it
// writes LDS, so their latencies overlap.
template <int LDP, int NTH = 256>
__device__ __forceinline__ void fill_upper(double (*S)[LDP], const double* __restrict__ M, int r, int ld,
                                           int tid) {
    constexpr int kFillPerThread = (kGaugeMaxRank * kGaugeMaxRank + NTH - 1) / NTH;
    double v[kFillPerThread];
#pragma unroll
    for (int q = 0; q < kFillPerThread; ++q) {
        const int idx = tid + q * NTH;
        const int i = idx / r, j = idx - i * r;
        v[q] = (idx < r * r && j >= i) ? M[(int64_t)i * ld + j] : 0.0;
    }
#pragma unroll
    for (int q = 0; q < kFillPerThread; ++q) {
        const int idx = tid + q * NTH;
        const int i = idx / r, j = idx - i * r;
        if (idx < r * r) S[i][j] = v[q];
    }
}

__global__ __launch_bounds__(kCholThreads) void k_gauge_chol(const double* __restrict__ G, int r, int ld,
                                                             double* __restrict__ R, int* __restrict__ flag,
                                                             double shift_rel) {
    __shared__ double S[kGaugeMaxRank][kGaugeMaxRank + 1];
    __shared__ double Rm[kGaugeMaxRank][kGaugeMaxRank + 1];   // R, written out at the end
    __shared__ double diag0[kGaugeMaxRank];
    __shared__ int bad;
    constexpr int kBlk = (kGaugeMaxRank + kCholSide - 1) / kCholSide;
    const int tid = threadIdx.x, tx = tid % kCholSide, ty = tid / kCholSide;
    fill_upper<kGaugeMaxRank + 1, kCholThreads>(S, G, r, ld, tid);
    if (tid == 0) bad = 0;
    __syncthreads();
    if (shift_rel > 0.0) {
        // trace summed by one thread in index order (deterministic)
        if (tid == 0) {
            double tr = 0.0;
            for (int i = 0; i < r; ++i) tr += S[i][i];
            const double sh = shift_rel * tr;
            for (int i = 0; i < r; ++i) S[i][i] += sh;
        }
        __syncthreads();
    }
    for (int i = tid; i < r; i += kCholThreads) diag0[i] = S[i][i];
    __syncthreads();
    for (int k = 0; k < r; ++k) {
        const double d = S[k][k];
        const double dk = d > 0.0 ? d : 0.0;
        const double sq = __builtin_sqrt(dk), inv = 1.0 / dk;
        if (tid == 0 && !(d > 0x1p-46 * diag0[k]) && bad == 0) bad = 1 + k;
        // row k of R (row k of S is not written in this step); global
        // stores here would make every barrier wait for them
        for (int j = k + tid; j < r; j += kCholThreads) Rm[k][j] = j == k ? sq : S[k][j] / sq;
        // trailing update of the upper triangle, k < i <= j: thread (ty, tx)
        // of the square thread grid takes rows ty + kCholSide a and columns
        // tx + kCholSide b;
        // each row's reads are issued together before its writes
        double rk[kBlk];
#pragma unroll
        for (int b = 0; b < kBlk; ++b) {
            const int j = b * kCholSide + tx;
            rk[b] = (j > k && j < r) ? S[k][j] : 0.0;
        }
#pragma unroll
        for (int a = 0; a < kBlk; ++a) {
            const int i = a * kCholSide + ty;
            if (i > k && i < r) {
                const double ski = S[k][i] * inv;
                double cur[kBlk];
#pragma unroll
                for (int b = 0; b < kBlk; ++b) {
                    const int j = b * kCholSide + tx;
                    cur[b] = (j >= i && j < r) ? S[i][j] : 0.0;
                }
#pragma unroll
                for (int b = 0; b < kBlk; ++b) {
                    const int j = b * kCholSide + tx;
                    if (j >= i && j < r) S[i][j] = cur[b] - ski * rk[b];
                }
            }
        }
        __syncthreads();
    }
    if (tid == 0 && bad) *flag = bad;
    for (int idx = tid; idx < ld * ld; idx += kCholThreads) {
        const int i = idx / ld, j = idx - i * ld;
        R[idx] = (i < r && j < r && j >= i) ? Rm[i][j] : 0.0;
    }
}

__device__ __forceinline__ double lane_value(double v, int lane) {
    const long long b = __builtin_bit_cast(long long, v);
    const int lo = __builtin_amdgcn_readlane((int)(b & 0xFFFFFFFFll), lane);
    const int hi = __builtin_amdgcn_readlane((int)(b >> 32), lane);
    return __builtin_bit_cast(double, ((long long)hi << 32) | (unsigned int)lo);
}

// C = A R^{-1} row by row (R upper triangular r x r with pitch ldr, A with
// pitch lda, C with pitch ldc whose pad columns r <= j < ldc are zeroed):
// forward substitution x R = a, x_t = a'_t / R[t][t], a'_j -= x_t R[t][j].
// One wave per group of kTrsmRows rows; lane j keeps a'_j (and, for TWO,
// that is r > 64, a'_{j+64}); the pivot value a'_t reaches the wave through
// a uniform readlane, and R sits in LDS, its next row read one step ahead.
// Lanes at or past r work on values that are never stored (R's entries
// there are not initialized), so the loop needs no masks.
constexpr int kTrsmRows = 4;
template <bool TWO>
__global__ __launch_bounds__(256) void k_gauge_trsm(const double* __restrict__ A, int64_t rows, int r, int lda,
                                                    const double* __restrict__ R, int ldr,
                                                    double* __restrict__ C, int ldc) {
    // one spare row and column: the prefetch of row t + 1 and the lanes
    // j + 64 < 128 stay inside the array
    __shared__ double Rs[kGaugeMaxRank + 1][kGaugeMaxRank + 1];
    __shared__ double inv[kGaugeMaxRank + 1];
    fill_upper(Rs, R, r, ldr, threadIdx.x);
    __syncthreads();
    for (int t = threadIdx.x; t < r; t += 256) inv[t] = 1.0 / Rs[t][t];
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const bool l0 = lane < r, l1 = lane + 64 < r;
    const int c1 = lane + 64 < kGaugeMaxRank + 1 ? lane + 64 : 0;   // column of a'_{j+64} (clamped)
    const int r0 = r < 64 ? r : 64;
    const int64_t w0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * kTrsmRows;
    const int64_t ws = (int64_t)gridDim.x * 4 * kTrsmRows;
    for (int64_t i0 = w0; i0 < rows; i0 += ws) {
        double a0[kTrsmRows], a1[kTrsmRows], x0[kTrsmRows], x1[kTrsmRows];
#pragma unroll
        for (int u = 0; u < kTrsmRows; ++u) {
            const int64_t i = i0 + u < rows ? i0 + u : rows - 1;
            const double* a = A + i * lda;
            a0[u] = l0 ? a[lane] : 0.0;
            a1[u] = (TWO && l1) ? a[lane + 64] : 0.0;
            x0[u] = x1[u] = 0.0;
        }
        double rt0 = Rs[0][lane], rt1 = TWO ? Rs[0][c1] : 0.0, it = inv[0];
        for (int t = 0; t < r0; ++t) {
            const double n0 = Rs[t + 1][lane];
            const double n1 = TWO ? Rs[t + 1][c1] : 0.0;
            const double nit = inv[t + 1];
#pragma unroll
            for (int u = 0; u < kTrsmRows; ++u) {
                const double xt = lane_value(a0[u], t) * it;
                x0[u] = lane == t ? xt : x0[u];
                a0[u] -= xt * rt0;
                if (TWO) a1[u] -= xt * rt1;
            }
            rt0 = n0;
            rt1 = n1;
            it = nit;
        }
        if (TWO) {
            rt1 = Rs[64][c1];
            it = inv[64];
            for (int t = 64; t < r; ++t) {
                const double n1 = Rs[t + 1][c1];
                const double nit = inv[t + 1];
#pragma unroll
                for (int u = 0; u < kTrsmRows; ++u) {
                    const double xt = lane_value(a1[u], t - 64) * it;
                    x1[u] = lane + 64 == t ? xt : x1[u];
                    a1[u] -= xt * rt1;
                }
                rt1 = n1;
                it = nit;
            }
        }
#pragma unroll
        for (int u = 0; u < kTrsmRows; ++u) {
            if (i0 + u >= rows) break;
            double* c = C + (i0 + u) * ldc;
            if (lane < ldc) c[lane] = l0 ? x0[u] : 0.0;
            if (lane + 64 < ldc) c[lane + 64] = l1 ? x1[u] : 0.0;
        }
    }
}

// C[i][c] = sum_{t >= i} R[i][t] X[t][c] for i < r, c < ncols (R upper
// triangular with pitch ldr, X and C r x ncols dense).  Workgroup (x, y)
// takes columns 256 x .. 256 x + 255 (one per thread, read coalesced) and
// output rows 32 y .. 32 y + 31, whose rows of R it keeps in LDS (zero
// below the diagonal, so the loop has no masks).
constexpr int kLmulRows = 32;
__global__ __launch_bounds__(256) void k_gauge_lmul(const double* __restrict__ R, int r, int ldr,
                                                    const double* __restrict__ X, int64_t ncols,
                                                    double* __restrict__ C) {
    __shared__ double Rs[LRC_GAUGE_MAX_RANK][kLmulRows];   // Rs[t][u] = R[i0 + u][t]
    const int i0 = blockIdx.y * kLmulRows;
    // all loads first, then the LDS writes (their latencies overlap)
    constexpr int kPer = LRC_GAUGE_MAX_RANK * kLmulRows / 256;
    double v[kPer];
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int idx = threadIdx.x + q * 256;
        const int t = idx / kLmulRows, i = i0 + idx % kLmulRows;
        v[q] = (t < r && i < r && t >= i) ? R[(int64_t)i * ldr + t] : 0.0;
    }
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
        const int idx = threadIdx.x + q * 256;
        Rs[idx / kLmulRows][idx % kLmulRows] = v[q];
    }
    __syncthreads();
    const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (c >= ncols) return;
    double acc[kLmulRows];
#pragma unroll
    for (int u = 0; u < kLmulRows; ++u) acc[u] = 0.0;
    // columns of X in batches of 8 rows: the loads of a batch overlap
    for (int t0 = i0; t0 < r; t0 += 8) {
        double xv[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) xv[q] = t0 + q < r ? X[(int64_t)(t0 + q) * ncols + c] : 0.0;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            if (t0 + q < r) {
#pragma unroll
                for (int u = 0; u < kLmulRows; ++u) acc[u] += Rs[t0 + q][u] * xv[q];
            }
        }
    }
#pragma unroll
    for (int u = 0; u < kLmulRows; ++u)
        if (i0 + u < r) C[(int64_t)(i0 + u) * ncols + c] = acc[u];
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
        b += round_up((int64_t)(rp * rp * 8), 256) * 3;                     // G, R1, R2
        b += round_up((int64_t)gram_workspace_bytes(rows, rp), 256);        // Gram partials
        b += round_up((int64_t)(r * ncols * 8), 256);                       // R1 G_{l+1}
        need = b > need ? b : need;
    }
    return need + 256 + (size_t)round_up(4 * (int64_t)d, 256);
}

__global__ void k_gauge_zero(int* p, int n) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

static unsigned trsm_grid(int64_t rows) {
    // enough waves to cover the rows in a few passes without reloading R
    // into LDS more often than needed
    int64_t g = (rows + 4 * kTrsmRows - 1) / (4 * kTrsmRows);
    if (g > 1024) g = 1024;
    return (unsigned)(g < 1 ? 1 : g);
}

static void launch_trsm(const double* A, int64_t rows, int r, int lda, const double* R, int ldr, double* C,
                        int ldc, hipStream_t stream) {
    if (r > 64)
        hipLaunchKernelGGL(k_gauge_trsm<true>, dim3(trsm_grid(rows)), dim3(256), 0, stream, A, rows, r, lda, R, ldr,
                           C, ldc);
    else
        hipLaunchKernelGGL(k_gauge_trsm<false>, dim3(trsm_grid(rows)), dim3(256), 0, stream, A, rows, r, lda, R,
                           ldr, C, ldc);
}

size_t cholqr2_workspace_bytes(int64_t rows, int r) {
    const int64_t rp = round_up(r, 2);
    return (size_t)round_up(rows * rp * 8, 256) + 5 * (size_t)round_up(rp * rp * 8, 256) +
           (size_t)round_up((int64_t)gram_workspace_bytes(rows, rp), 256);
}

hipError_t launch_cholqr2(const double* A, int64_t rows, int r, double* Q, double* R, int* flag, Workspace& ws,
                          hipStream_t stream, const char* label, bool shifted) {
    const int rp = (int)round_up(r, 2);
    double* W2 = static_cast<double*>(ws.take((size_t)rows * rp * 8));
    double* G = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    double* R1 = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    double* R2 = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    double* R3 = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    double* RX = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    if (ws.overrun) return hipErrorOutOfMemory;
    KernelTimer tm(label, stream);
    const size_t gmark = ws.used;
    // one pass: Gram of `in`, its Cholesky factor `Rk`, out = in Rk^{-1}
    auto pass = [&](const double* in, double* Rk, double* out, double shift_rel) {
        hipError_t e = launch_gram(in, rows, rp, G, ws, stream);
        ws.used = gmark;
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(k_gauge_chol, dim3(1), dim3(kCholThreads), 0, stream, G, r, rp, Rk, flag, shift_rel);
        launch_trsm(in, rows, r, rp, Rk, rp, out, rp, stream);
        return hipGetLastError();
    };
    // rows 0..r-1 of the triangular product dst = Ra Rb (Rb taken as an r x rp block)
    auto tri = [&](const double* Ra, const double* Rb, double* dst) {
        const dim3 gl((unsigned)((rp + 255) / 256), (unsigned)((r + kLmulRows - 1) / kLmulRows));
        hipLaunchKernelGGL(k_gauge_lmul, gl, dim3(256), 0, stream, Ra, r, rp, Rb, (int64_t)rp, dst);
    };
    hipError_t e;
    if (!shifted) {
        if ((e = pass(A, R1, W2, 0.0)) != hipSuccess || (e = pass(W2, R2, Q, 0.0)) != hipSuccess) return e;
        if (R) tri(R2, R1, R);
    } else {
        // shifted CholeskyQR3 (Fukaya, Kannan, Nakatsukasa, Yamamoto, Yanagisawa 2020): the shift
        // s = 11 (m r + r (r + 1)) u ||A||_F^2 keeps the first factorization away from breakdown for
        // condition numbers up to about u^-1; two plain passes restore orthogonality
        const double shift_rel = 11.0 * ((double)rows * r + (double)r * (r + 1)) * 0x1p-53;
        if ((e = pass(A, R1, Q, shift_rel)) != hipSuccess || (e = pass(Q, R2, W2, 0.0)) != hipSuccess ||
            (e = pass(W2, R3, Q, 0.0)) != hipSuccess)
            return e;
        if (R) {
            tri(R2, R1, RX);
            tri(R3, RX, R);
        }
    }
    return hipGetLastError();
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
        double* R2 = static_cast<double*>(ws.take((size_t)rp * rp * 8));
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
        hipLaunchKernelGGL(k_gauge_chol, dim3(1), dim3(kCholThreads), 0, stream, G, r, rp, R1, flags + l, 0.0);
        launch_trsm(W1, rows, r, rp, R1, rp, W2, rp, stream);
        // second pass on W2: core l = W2 R2^{-1}; R = R2 R1
        e = launch_gram(W2, rows, rp, G, ws, stream);
        if (e != hipSuccess) return e;
        ws.used = gmark;
        hipLaunchKernelGGL(k_gauge_chol, dim3(1), dim3(kCholThreads), 0, stream, G, r, rp, R2, flags + l, 0.0);
        launch_trsm(W2, rows, r, rp, R2, rp, cores[l], r, stream);
        // core l+1 <- R2 (R1 core l+1) on its left unfolding (r x ncols)
        const dim3 gl((unsigned)((ncols + 255) / 256), (unsigned)((r + kLmulRows - 1) / kLmulRows));
        hipLaunchKernelGGL(k_gauge_lmul, gl, dim3(256), 0, stream, R1, r, rp, cores[l + 1], ncols, NX);
        hipLaunchKernelGGL(k_gauge_lmul, gl, dim3(256), 0, stream, R2, r, rp, NX, ncols, cores[l + 1]);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        ws.used = mark;
    }
    return hipSuccess;
}

}  // namespace lrc

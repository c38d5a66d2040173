// Randomized FP64 factorizations on the device: the end-to-end decomposition
// that Sec. sec:conclusion leaves to future work, so that a dense matrix or
// tensor can be factored where the rank-compensated factors are then
// stored, applied and certified.  The method is the randomized range finder
// of Halko, Martinsson and Tropp (SIAM Review 2011) with the exact SVD of the
// small projected matrix, and TT-SVD (Sec. 5.1) with every truncated SVD
// replaced by it.  The Gaussian test vectors are inputs.
//
// Matrix A (m x n), l test vectors as the rows of Omega (l x n):
//   Y = A Omega^T                 split-K MFMA GEMM (m x l)
//   Y = Q R_Y                     CholeskyQR2 (Q^T Q = I)
//   q times: Z = orth(A^T Q), Q = orth(A Z)
//   B^T = A^T Q = Q_2 R           MFMA GEMM (n x l), CholeskyQR2
//   R^T = W diag(sigma) Z^T       one-sided Jacobi in one workgroup (l x l)
//   U = Q W,  V = Q_2 Z           (A ~= Q B = Q R^T Q_2^T = U diag(sigma) V^T)
// Only the GEMMs over A touch more than O((m + n) l) data; they run on the
// FP64 matrix cores and bound the whole (2 m n l flop each).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "../../include/lrc.h"
#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

constexpr int kFactMaxL = LRC_RSVD_MAX_SAMPLES;
constexpr int kJacThreads = 1024;
constexpr int kJacWaves = kJacThreads / 64;
constexpr int kJacSweeps = 40;

// dst (drows x ldd) = src (rows x cols, pitch lds) with zeros past rows / cols
__global__ __launch_bounds__(256) void k_fact_pad(const double* __restrict__ src, int64_t rows, int64_t cols,
                                                  int64_t lds, double* __restrict__ dst, int64_t drows, int64_t ldd) {
    const int64_t total = drows * ldd;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total; idx += (int64_t)gridDim.x * 256) {
        const int64_t i = idx / ldd, j = idx - i * ldd;
        dst[idx] = (i < rows && j < cols) ? src[i * lds + j] : 0.0;
    }
}

// dst[j][i] = src[i][j] (src rows x cols with pitch lds; dst cols x ldd),
// zero for rows <= i < ldd; 32 x 32 tiles through LDS.
__global__ __launch_bounds__(256) void k_fact_transpose(const double* __restrict__ src, int64_t rows, int64_t cols,
                                                        int64_t lds, double* __restrict__ dst, int64_t ldd) {
    __shared__ double tile[32][33];
    const int64_t i0 = (int64_t)blockIdx.x * 32, j0 = (int64_t)blockIdx.y * 32;
    const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;
    for (int u = ty; u < 32; u += 8) {
        const int64_t i = i0 + u, j = j0 + tx;
        tile[u][tx] = (i < rows && j < cols) ? src[i * lds + j] : 0.0;
    }
    __syncthreads();
    for (int u = ty; u < 32; u += 8) {
        const int64_t j = j0 + u, i = i0 + tx;
        if (j < cols && i < ldd) dst[j * ldd + i] = tile[tx][u];
    }
}

__global__ void k_fact_zero(int* p, int n) {
    for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = 0;
}

// Value of lane `ctl` (a DPP row permutation) for a double: its two halves
// moved by the same data-parallel-primitive move.
template <int CTL>
__device__ __forceinline__ double dpp_f64(double v) {
    const long long b = __builtin_bit_cast(long long, v);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(b & 0xFFFFFFFFll), CTL, 0xF, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(b >> 32), CTL, 0xF, 0xF, false);
    return __builtin_bit_cast(double, ((long long)hi << 32) | (unsigned int)lo);
}

// Sums of three values over each group of 16 lanes: butterfly by lane
// swaps within quads (xor 1, xor 2), then the mirror within each half row
// (lane i with 7 - i) and within the row (i with 15 - i).  Each step adds
// two equal-ordered partial sums, so all 16 lanes end with identical
// totals (branches on them stay uniform within the group).
__device__ __forceinline__ void group16_sum3(double& a, double& b, double& c) {
    constexpr int kXor1 = 0xB1, kXor2 = 0x4E, kHalfMirror = 0x141, kMirror = 0x140;
    a += dpp_f64<kXor1>(a); b += dpp_f64<kXor1>(b); c += dpp_f64<kXor1>(c);
    a += dpp_f64<kXor2>(a); b += dpp_f64<kXor2>(b); c += dpp_f64<kXor2>(c);
    a += dpp_f64<kHalfMirror>(a); b += dpp_f64<kHalfMirror>(b); c += dpp_f64<kHalfMirror>(c);
    a += dpp_f64<kMirror>(a); b += dpp_f64<kMirror>(b); c += dpp_f64<kMirror>(c);
}

// One workgroup: SVD of M = R^T (R upper triangular, l x l inside pitch ldr)
// by one-sided (Hestenes) Jacobi.  The columns of M (rows of R) and of the
// accumulated rotation Z sit in LDS, the columns first put in non-increasing
// order of their norms (de Rijk's ordering); a sweep visits every column pair once
// in l' - 1 rounds of the round-robin (circle) ordering, l' = l rounded up to
// even.  The l'/2 <= 48 disjoint pairs of a round run at once, one per
// group of 16 lanes (64 groups), each lane holding entries e = lane + 16 u
// of the two columns.  A pair (p, q) is rotated when |m_p . m_q| > tol
// ||m_p|| ||m_q||, tol = max(l, 8) 2^-53, by the rotation that makes the two
// columns orthogonal (the smaller root of t^2 + 2 zeta t - 1 = 0, zeta =
// (|m_q|^2 - |m_p|^2) / (2 m_p . m_q)).  The sweeps stop when one rotates
// nothing; *flag = 1 if 40 sweeps do not get there.  Then sigma_j = ||m_j||,
// and the columns are written in non-increasing order of sigma (ties by
// index): sv[pos] = sigma, Wt[pos][:] = m_j / sigma_j (zero when sigma_j =
// 0), Zt[pos][:] = z_j, and, when Zts is not null, Zts[pos][:] = sigma_j z_j;
// rows of pitch ldw with zeros in columns l..ldw-1; s_out[pos] = sigma for
// pos < k when not null.
constexpr int kJacPer = kFactMaxL / 16;   // entries of a column per lane
static_assert(kFactMaxL % 16 == 0 && kFactMaxL / 2 <= kJacThreads / 16, "one group of 16 lanes per pair");
__global__ __launch_bounds__(kJacThreads) void k_fact_jacobi(const double* __restrict__ R, int l, int ldr, int k,
                                                             double* __restrict__ sv, double* __restrict__ s_out,
                                                             double* __restrict__ Wt, double* __restrict__ Zt,
                                                             double* __restrict__ Zts, int ldw, int* __restrict__ flag) {
    __shared__ double Mc[kFactMaxL][kFactMaxL + 1];
    __shared__ double Jc[kFactMaxL][kFactMaxL + 1];
    __shared__ double sig[kFactMaxL];
    __shared__ int pos[kFactMaxL];
    __shared__ int rotated;
    const int tid = threadIdx.x;
    const int grp = tid >> 4, gl = tid & 15;
    // columns of M = R^T (rows of R) placed in non-increasing order of their
    // norms (ties by index), which shortens the sweeps; the rotation
    // accumulator starts as that permutation
    for (int j = grp; j < l; j += kJacThreads / 16) {
        double x = 0.0, y = 0.0, z = 0.0;
#pragma unroll
        for (int u = 0; u < kJacPer; ++u) {
            const int e = gl + 16 * u;
            const double v = (e < l && e >= j) ? R[(int64_t)j * ldr + e] : 0.0;
            x += v * v;
        }
        group16_sum3(x, y, z);
        if (gl == 0) sig[j] = x;
    }
    __syncthreads();
    if (tid < l) {
        const double sj = sig[tid];
        int c = 0;
        for (int i = 0; i < l; ++i) c += (sig[i] > sj || (sig[i] == sj && i < tid)) ? 1 : 0;
        pos[tid] = c;
    }
    __syncthreads();
    for (int idx = tid; idx < l * l; idx += kJacThreads) {
        const int j = idx / l, i = idx - j * l;
        Mc[pos[j]][i] = i >= j ? R[(int64_t)j * ldr + i] : 0.0;
        Jc[pos[j]][i] = i == j ? 1.0 : 0.0;
    }
    if (tid == 0) rotated = 0;
    __syncthreads();
    const int L = l + (l & 1);
    const double tol = (double)(l > 8 ? l : 8) * 0x1p-53;
    bool converged = false;
    for (int sweep = 0; sweep < kJacSweeps; ++sweep) {
        int a = grp, b = L - 1;   // round 0's pair of this group (pair s = grp)
        for (int t = 0; t + 1 < L; ++t) {
            if (grp < L / 2) {
                if (grp == 0) {
                    a = t;
                    b = L - 1;
                } else {
                    a = t + grp;
                    a = a >= L - 1 ? a - (L - 1) : a;
                    b = t - grp;
                    b = b < 0 ? b + (L - 1) : b;
                }
                const int p = a < b ? a : b, q = a < b ? b : a;
                if (q < l) {
                    double mp[kJacPer], mq[kJacPer];
                    double al = 0.0, be = 0.0, ga = 0.0;
#pragma unroll
                    for (int u = 0; u < kJacPer; ++u) {
                        const int e = gl + 16 * u;
                        mp[u] = e < l ? Mc[p][e] : 0.0;
                        mq[u] = e < l ? Mc[q][e] : 0.0;
                        al += mp[u] * mp[u];
                        be += mq[u] * mq[u];
                        ga += mp[u] * mq[u];
                    }
                    group16_sum3(al, be, ga);
                    if (ga != 0.0 && __builtin_fabs(ga) > tol * __builtin_sqrt(al) * __builtin_sqrt(be)) {
                        const double zeta = (be - al) / (2.0 * ga);
                        const double az = __builtin_fabs(zeta);
                        double tt = az > 1e150 ? 0.5 / az : 1.0 / (az + __builtin_sqrt(1.0 + zeta * zeta));
                        tt = zeta < 0.0 ? -tt : tt;
                        const double c = 1.0 / __builtin_sqrt(1.0 + tt * tt), sn = c * tt;
#pragma unroll
                        for (int u = 0; u < kJacPer; ++u) {
                            const int e = gl + 16 * u;
                            if (e < l) {
                                Mc[p][e] = c * mp[u] - sn * mq[u];
                                Mc[q][e] = sn * mp[u] + c * mq[u];
                                const double jp = Jc[p][e], jq = Jc[q][e];
                                Jc[p][e] = c * jp - sn * jq;
                                Jc[q][e] = sn * jp + c * jq;
                            }
                        }
                        if (gl == 0) rotated = 1;
                    }
                }
            }
            __syncthreads();
        }
        const bool any = rotated != 0;
        __syncthreads();   // every thread has read the flag
        if (tid == 0) rotated = 0;
        __syncthreads();   // the reset lands before the next sweep's rotations
        if (!any) {
            converged = true;
            break;
        }
    }
    if (tid == 0 && !converged) *flag = 1;
    // singular values: one group of 16 lanes per column
    for (int j = grp; j < l; j += kJacThreads / 16) {
        double x = 0.0, y = 0.0, z = 0.0;
#pragma unroll
        for (int u = 0; u < kJacPer; ++u) {
            const int e = gl + 16 * u;
            const double v = e < l ? Mc[j][e] : 0.0;
            x += v * v;
        }
        group16_sum3(x, y, z);
        if (gl == 0) sig[j] = __builtin_sqrt(x);
    }
    __syncthreads();
    if (tid < l) {
        const double sj = sig[tid];
        int c = 0;
        for (int i = 0; i < l; ++i) c += (sig[i] > sj || (sig[i] == sj && i < tid)) ? 1 : 0;
        pos[tid] = c;
        sv[c] = sj;
        if (s_out && c < k) s_out[c] = sj;
    }
    __syncthreads();
    for (int idx = tid; idx < l * ldw; idx += kJacThreads) {
        const int j = idx / ldw, e = idx - j * ldw;
        const double sj = sig[j];
        const int64_t o = (int64_t)pos[j] * ldw + e;
        const double m = e < l ? Mc[j][e] : 0.0, z = e < l ? Jc[j][e] : 0.0;
        Wt[o] = sj > 0.0 ? m / sj : 0.0;
        Zt[o] = z;
        if (Zts) Zts[o] = sj * z;
    }
}

static unsigned fact_grid(int64_t items) {
    int64_t g = (items + 255) / 256;
    if (g > 8192) g = 8192;
    return (unsigned)(g < 1 ? 1 : g);
}

static size_t r256(int64_t bytes) { return (size_t)round_up(bytes, 256); }

size_t rsvd_workspace_bytes(int64_t m, int64_t n, int l, int k, int q, bool vts) {
    const int64_t rp = round_up(l, 2), ldn = round_up(n, 2);
    size_t keep = 2 * r256(m * rp * 8) + 2 * r256(n * rp * 8) + 4 * r256(rp * rp * 8) + r256(rp * 8);
    if (q > 0) keep += r256(rp * ldn * 8);
    size_t tmp = gemm_nt_workspace_bytes(l, m, n);
    tmp = std::max(tmp, gemm_tn_workspace_bytes(l, n, m));
    tmp = std::max(tmp, cholqr2_workspace_bytes(m, l));
    tmp = std::max(tmp, cholqr2_workspace_bytes(n, l));
    tmp = std::max(tmp, gemm_nt_workspace_bytes(k, m, l));
    tmp = std::max(tmp, gemm_nt_workspace_bytes(k, n, l));
    if (vts) tmp = std::max(tmp, gemm_nt_workspace_bytes(n, k, l));
    return keep + tmp + 4096;
}

// A (m x n, pitch lda) and Omega (l x n, pitch ldo): 16-byte aligned, even
// pitches.  Outputs (any that are null are skipped): U (m x k, pitch ldu),
// s_out (k), V (n x k, pitch ldv), Vts = diag(s) V^T (k x n, pitch ldvt).
// flags[0]: range finder QR, flags[1]: QR of B^T, flags[2]: Jacobi.
// shifted: every orthonormalization by shifted CholeskyQR3 instead of
// CholeskyQR2 (for sketches with condition numbers between about 1e7 and
// 1e15; half as much QR work again).
hipError_t launch_rsvd(const double* A, int64_t m, int64_t n, int64_t lda, const double* Om, int64_t ldo, int l,
                       int q, int k, double* U, int64_t ldu, double* s_out, double* V, int64_t ldv, double* Vts,
                       int64_t ldvt, int* flags, Workspace& ws, hipStream_t st, bool shifted) {
    const int rp = (int)round_up(l, 2);
    const int64_t ldn = round_up(n, 2);
    double* Y = static_cast<double*>(ws.take((size_t)m * rp * 8));
    double* Q = static_cast<double*>(ws.take((size_t)m * rp * 8));
    double* Bt = static_cast<double*>(ws.take((size_t)n * rp * 8));
    double* Q2 = static_cast<double*>(ws.take((size_t)n * rp * 8));
    double* R = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    double* Wt = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    double* Zt = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    double* Zs = static_cast<double*>(ws.take((size_t)rp * rp * 8));
    double* sv = static_cast<double*>(ws.take((size_t)rp * 8));
    double* Qzt = q > 0 ? static_cast<double*>(ws.take((size_t)rp * ldn * 8)) : nullptr;
    if (ws.overrun) return hipErrorOutOfMemory;
    const size_t mark = ws.used;
    hipError_t e;
#define LRC_STEP(call)                     \
    do {                                   \
        e = (call);                        \
        if (e != hipSuccess) return e;     \
        ws.used = mark;                    \
    } while (0)
    LRC_STEP(launch_gemm_nt(Om, ldo, l, A, lda, m, n, nullptr, Y, rp, rp, ws, st, "factor_sketch_f64"));
    LRC_STEP(launch_cholqr2(Y, m, l, Q, nullptr, flags, ws, st, "factor_cholqr2_f64", shifted));
    for (int it = 0; it < q; ++it) {
        LRC_STEP(launch_gemm_tn(Q, rp, l, A, lda, n, m, Bt, rp, rp, ws, st, "factor_project_f64",
                                "factor_project_finish_f64"));
        LRC_STEP(launch_cholqr2(Bt, n, l, Q2, nullptr, flags, ws, st, "factor_cholqr2_f64", shifted));
        {
            KernelTimer tm("factor_transpose_f64", st);
            hipLaunchKernelGGL(k_fact_transpose, dim3((unsigned)((ldn + 31) / 32), (unsigned)((rp + 31) / 32)),
                               dim3(256), 0, st, Q2, n, (int64_t)rp, (int64_t)rp, Qzt, ldn);
        }
        LRC_STEP(launch_gemm_nt(Qzt, ldn, l, A, lda, m, n, nullptr, Y, rp, rp, ws, st, "factor_sketch_f64"));
        LRC_STEP(launch_cholqr2(Y, m, l, Q, nullptr, flags, ws, st, "factor_cholqr2_f64", shifted));
    }
    LRC_STEP(launch_gemm_tn(Q, rp, l, A, lda, n, m, Bt, rp, rp, ws, st, "factor_project_f64",
                            "factor_project_finish_f64"));
    LRC_STEP(launch_cholqr2(Bt, n, l, Q2, R, flags + 1, ws, st, "factor_cholqr2_f64", shifted));
    {
        KernelTimer tm("factor_jacobi_f64", st);
        hipLaunchKernelGGL(k_fact_jacobi, dim3(1), dim3(kJacThreads), 0, st, R, l, rp, k, sv, s_out, Wt, Zt,
                           Vts ? Zs : nullptr, rp, flags + 2);
    }
    if (U) LRC_STEP(launch_gemm_nt(Wt, rp, k, Q, rp, m, l, nullptr, U, ldu, k, ws, st, "factor_vectors_f64"));
    if (V) LRC_STEP(launch_gemm_nt(Zt, rp, k, Q2, rp, n, l, nullptr, V, ldv, k, ws, st, "factor_vectors_f64"));
    if (Vts) LRC_STEP(launch_gemm_nt(Q2, rp, n, Zs, rp, k, l, nullptr, Vts, ldvt, n, ws, st, "factor_vectors_f64"));
#undef LRC_STEP
    return hipGetLastError();
}

// Padded copy (rows x cols -> rows x even pitch) when the source is not fit
// for 16-byte moves; returns the pointer and pitch to use.
static hipError_t fit(const double* src, int64_t rows, int64_t cols, Workspace& ws, hipStream_t st,
                      const double** out, int64_t* ld) {
    if (cols % 2 == 0 && reinterpret_cast<uintptr_t>(src) % 16 == 0) {
        *out = src;
        *ld = cols;
        return hipSuccess;
    }
    const int64_t p = round_up(cols, 2);
    double* d = static_cast<double*>(ws.take((size_t)rows * p * 8));
    if (ws.overrun) return hipErrorOutOfMemory;
    KernelTimer tm("factor_pad_f64", st);
    hipLaunchKernelGGL(k_fact_pad, dim3(fact_grid(rows * p)), dim3(256), 0, st, src, rows, cols, cols, d, rows, p);
    *out = d;
    *ld = p;
    return hipGetLastError();
}

static size_t fit_bytes(int64_t rows, int64_t cols) { return r256(rows * round_up(cols, 2) * 8); }

size_t matrix_rsvd_workspace_bytes(int64_t m, int64_t n, int l, int k, int q) {
    return 3 * 256 + fit_bytes(m, n) + fit_bytes(l, n) + rsvd_workspace_bytes(m, n, l, k, q, false);
}

hipError_t launch_matrix_rsvd(const double* A, int64_t m, int64_t n, const double* Om, int l, int q, int k, double* U,
                              double* s, double* V, int* flags, Workspace& ws, hipStream_t st, bool shifted) {
    hipLaunchKernelGGL(k_fact_zero, dim3(1), dim3(64), 0, st, flags, 3);
    const double *Af, *Of;
    int64_t lda, ldo;
    hipError_t e = fit(A, m, n, ws, st, &Af, &lda);
    if (e == hipSuccess) e = fit(Om, l, n, ws, st, &Of, &ldo);
    if (e != hipSuccess) return e;
    return launch_rsvd(Af, m, n, lda, Of, ldo, l, q, k, U, k, s, V, k, nullptr, 0, flags, ws, st, shifted);
}

// TT-SVD, step l of d - 1: C_l ((r_{l-1} n_l) x prod_{i>l} n_i) -> core l =
// U (pitch r_l), C_{l+1} = diag(s) V^T (r_l x cols, contiguous, which is
// C_{l+1} reshaped); the last step writes diag(s) V^T into the last core.
size_t tt_rsvd_workspace_bytes(const int64_t* dims, const int64_t* ranks, const int64_t* samples, int d, int q) {
    size_t need = 0, cbuf = 0;
    int64_t cols = 1;
    for (int i = 1; i < d; ++i) cols *= dims[i];
    for (int l = 0; l + 1 < d; ++l) {
        const int64_t rows = ranks[l] * dims[l];
        size_t b = fit_bytes(rows, cols) + fit_bytes(samples[l], cols) +
                   rsvd_workspace_bytes(rows, cols, (int)samples[l], (int)ranks[l + 1], q, true);
        need = std::max(need, b);
        if (l + 2 < d) cbuf = std::max(cbuf, r256(ranks[l + 1] * cols * 8));
        cols /= dims[l + 1];
    }
    return need + 2 * cbuf + r256(4 * 3 * (int64_t)d) + 1024;
}

hipError_t launch_tt_rsvd(const double* T, const int64_t* dims, const int64_t* ranks, const int64_t* samples, int d,
                          const double* const* omegas, int q, double* const* cores, double* sigma, int* flags,
                          Workspace& ws, hipStream_t st, bool shifted) {
    hipLaunchKernelGGL(k_fact_zero, dim3(1), dim3(64), 0, st, flags, 3 * (d - 1));
    int64_t cols = 1;
    for (int i = 1; i < d; ++i) cols *= dims[i];
    size_t cbuf = 0;
    {
        int64_t c = cols;
        for (int l = 0; l + 2 < d; ++l) {
            cbuf = std::max(cbuf, (size_t)(ranks[l + 1] * c * 8));
            c /= dims[l + 1];
        }
    }
    double* Cb[2] = {nullptr, nullptr};
    if (cbuf) {
        Cb[0] = static_cast<double*>(ws.take(cbuf));
        Cb[1] = static_cast<double*>(ws.take(cbuf));
        if (ws.overrun) return hipErrorOutOfMemory;
    }
    const double* C = T;
    int64_t soff = 0;
    for (int l = 0; l + 1 < d; ++l) {
        const int64_t rows = ranks[l] * dims[l];
        const int r = (int)ranks[l + 1];
        const bool last = l + 2 == d;
        double* next = last ? cores[d - 1] : Cb[l & 1];
        const size_t mark = ws.used;
        const double *Af, *Of;
        int64_t lda, ldo;
        hipError_t e = fit(C, rows, cols, ws, st, &Af, &lda);
        if (e == hipSuccess) e = fit(omegas[l], samples[l], cols, ws, st, &Of, &ldo);
        if (e == hipSuccess)
            e = launch_rsvd(Af, rows, cols, lda, Of, ldo, (int)samples[l], q, r, cores[l], r,
                            sigma ? sigma + soff : nullptr, nullptr, 0, next, cols, flags + 3 * l, ws, st, shifted);
        if (e != hipSuccess) return e;
        ws.used = mark;
        soff += r;
        C = next;
        cols /= dims[l + 1];
    }
    return hipSuccess;
}

}  // namespace lrc

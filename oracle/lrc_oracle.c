/*
 * CPU oracle for low-precision rank compensation (El Mountasser & Jbilou,
 * "Low-Precision Rank Compensation for Matrices and Tensor Trains").
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain reference that the
 * GPU library is checked against.  Only the test suite, the smoke check and
 * the CPU-baseline leg of the benchmark may load it.  It shares no code,
 * header, table or helper with the GPU library.
 *
 * Everything is IEEE binary64, built with -ffp-contract=off and without
 * fast-math, so every function below is bitwise deterministic for any number
 * of OpenMP threads: threads only split independent output rows, and every
 * sum runs in ascending index order.
 *
 * Contents (each cites the passage it follows):
 *   - rounding of stored values to binary32 / binary16 (Sec. 3.2 formats,
 *     Remark after Thm 4.1: factors rounded individually);
 *   - the factor apply Y = U diag(s) V^T X (Sec. 4.4, eq. gpu_matrix_apply);
 *   - the TT reshape chain and the per-entry slice product (Sec. 5.1;
 *     Sec. 7.5, eq. gpu_tt_reconstruction; Sec. 3.4 independent evaluator);
 *   - Householder QR and one-sided Jacobi SVD for the offline factorizations
 *     (Sec. 4.3 FP64 SVD; Sec. 5.1 TT-SVD; Sec. 6.1 orthogonal gauge);
 *   - Frobenius sums of squares (Sec. 5.1 norm definition).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Rounding (Sec. 3.2, Table tab:precision_comparison_prelim: binary16 has 11
 * significand bits and 5 exponent bits; round-to-nearest, ties to even).    */
/* ------------------------------------------------------------------------ */

/* binary64 -> binary16 with ONE rounding step, ties to even, subnormals kept.
 * Returns the number of finite inputs that overflowed to +-inf.  Never goes
 * through binary32 (that would round twice). */
int64_t orc_round_f16(const double* x, uint16_t* h, int64_t n)
{
    int64_t overflow = 0;
    for (int64_t idx = 0; idx < n; ++idx) {
        double v = x[idx];
        uint16_t sign = signbit(v) ? 0x8000u : 0u;
        double a = fabs(v);
        if (isnan(v)) { h[idx] = (uint16_t)(sign | 0x7E00u); continue; }
        if (isinf(v)) { h[idx] = (uint16_t)(sign | 0x7C00u); continue; }
        /* The largest finite binary16 is 65504 = (2 - 2^-10) 2^15; the value
         * halfway to 2^16 is 65520, which ties to the even neighbour 2^16,
         * i.e. overflows. */
        if (a >= 65520.0) { h[idx] = (uint16_t)(sign | 0x7C00u); ++overflow; continue; }
        if (a < ldexp(1.0, -14)) {
            /* subnormal range: quantum 2^-24; q in [0, 1024] (1024 is the
             * smallest normal, whose encoding 0x0400 equals q). */
            double q = rint(ldexp(a, 24));
            h[idx] = (uint16_t)(sign | (uint16_t)q);
            continue;
        }
        int e2;
        (void)frexp(a, &e2);           /* a in [2^(e2-1), 2^e2) */
        int E = e2 - 1;                /* unbiased exponent, -14..15 */
        double q = rint(ldexp(a, 10 - E));  /* in [1024, 2048] */
        if (q == 2048.0) { q = 1024.0; E += 1; }
        if (E > 15) { h[idx] = (uint16_t)(sign | 0x7C00u); ++overflow; continue; }
        h[idx] = (uint16_t)(sign | (uint16_t)((E + 15) << 10) | (uint16_t)((int)q - 1024));
    }
    return overflow;
}

/* binary16 -> binary64, exact. */
void orc_f16_to_f64(const uint16_t* h, double* x, int64_t n)
{
    for (int64_t idx = 0; idx < n; ++idx) {
        uint16_t b = h[idx];
        int s = (b >> 15) & 1, e = (b >> 10) & 0x1F, f = b & 0x3FF;
        double v;
        if (e == 0) v = ldexp((double)f, -24);
        else if (e == 31) v = f ? NAN : INFINITY;
        else v = ldexp((double)(1024 + f), e - 25);
        x[idx] = s ? -v : v;
    }
}

/* binary64 -> binary32: the C conversion is correctly rounded in the default
 * round-to-nearest-even mode (subnormals and overflow included).  Returns the
 * number of finite inputs that overflowed. */
int64_t orc_round_f32(const double* x, float* y, int64_t n)
{
    int64_t overflow = 0;
    for (int64_t idx = 0; idx < n; ++idx) {
        float f = (float)x[idx];
        if (isinf(f) && !isinf(x[idx])) ++overflow;
        y[idx] = f;
    }
    return overflow;
}

/* ------------------------------------------------------------------------ */
/* Factor apply (Sec. 4.4, eq. gpu_matrix_apply, written with X as n x b):
 *   T[j][c]  = sum_i V[i][j] X[i][c]        (i ascending)
 *   T'[j][c] = s[j] T[j][c]
 *   Y[i][c]  = sum_j U[i][j] T'[j][c]       (j ascending)
 * U is m x k, V is n x k, X is n x b, Y is m x b, all row-major.           */
/* ------------------------------------------------------------------------ */
void orc_apply(const double* U, const double* s, const double* V, const double* X,
               double* Y, int64_t m, int64_t n, int64_t k, int64_t b)
{
    double* T = (double*)calloc((size_t)(k * b > 0 ? k * b : 1), sizeof(double));
    #pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < k; ++j) {
        double* trow = T + j * b;
        for (int64_t i = 0; i < n; ++i) {
            double vij = V[i * k + j];
            const double* xrow = X + i * b;
            for (int64_t c = 0; c < b; ++c) trow[c] += vij * xrow[c];
        }
        for (int64_t c = 0; c < b; ++c) trow[c] = s[j] * trow[c];
    }
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double* yrow = Y + i * b;
        for (int64_t c = 0; c < b; ++c) yrow[c] = 0.0;
        for (int64_t j = 0; j < k; ++j) {
            double uij = U[i * k + j];
            const double* trow = T + j * b;
            for (int64_t c = 0; c < b; ++c) yrow[c] += uij * trow[c];
        }
    }
    free(T);
}

/* Dense reconstruction A_r = U diag(s) V^T (m x n), the FP64 contraction
 * used for error measurement (Remark after Thm 4.1):
 *   A[i][j] = sum_t (U[i][t] s[t]) V[j][t],  t ascending. */
void orc_lowrank_dense(const double* U, const double* s, const double* V,
                       double* A, int64_t m, int64_t n, int64_t k)
{
    /* V^T copy so the innermost loop runs over contiguous memory */
    double* Vt = (double*)malloc((size_t)(k * n > 0 ? k * n : 1) * sizeof(double));
    for (int64_t j = 0; j < n; ++j)
        for (int64_t t = 0; t < k; ++t) Vt[t * n + j] = V[j * k + t];
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double* arow = A + i * n;
        for (int64_t j = 0; j < n; ++j) arow[j] = 0.0;
        for (int64_t t = 0; t < k; ++t) {
            double ut = U[i * k + t] * s[t];
            const double* vrow = Vt + t * n;
            for (int64_t j = 0; j < n; ++j) arow[j] += ut * vrow[j];
        }
    }
    free(Vt);
}

/* ------------------------------------------------------------------------ */
/* Tensor-Train evaluation (Sec. 5.1; Sec. 7.5 eq. gpu_tt_reconstruction).  */
/* cores[l] is r_l x n_l x r_{l+1} row-major, ranks[0] = ranks[d] = 1.      */
/* ------------------------------------------------------------------------ */

/* Reshape chain: Z_1 = G_1 as n_1 x r_1; B_l = Z_{l-1} K_l with K_l = G_l as
 * r_{l-1} x (n_l r_l); Z_l = B_l read as (n_1..n_l) x r_l.  The final buffer
 * (r_d = 1) is the C-order vectorized tensor, written to `out`. */
int orc_tt_chain(const double* const* cores, const int64_t* dims, const int64_t* ranks,
                 int d, double* out)
{
    if (d < 1) return -1;
    int64_t rows = dims[0];
    int64_t maxsz = dims[0] * ranks[1];
    int64_t p = dims[0];
    for (int l = 1; l < d; ++l) {
        p *= dims[l];
        int64_t sz = p * ranks[l + 1];
        if (sz > maxsz) maxsz = sz;
    }
    if (d == 1) {
        memcpy(out, cores[0], (size_t)dims[0] * sizeof(double));
        return 0;
    }
    double* za = (double*)malloc((size_t)maxsz * sizeof(double));
    double* zb = (double*)malloc((size_t)maxsz * sizeof(double));
    if (!za || !zb) { free(za); free(zb); return -2; }
    memcpy(za, cores[0], (size_t)(dims[0] * ranks[1]) * sizeof(double));
    for (int l = 1; l < d; ++l) {
        int64_t rin = ranks[l], cols = dims[l] * ranks[l + 1];
        const double* K = cores[l];
        double* dst = (l == d - 1) ? out : zb;
        #pragma omp parallel for schedule(static)
        for (int64_t r = 0; r < rows; ++r) {
            double* brow = dst + r * cols;
            const double* zrow = za + r * rin;
            for (int64_t q = 0; q < cols; ++q) brow[q] = 0.0;
            for (int64_t t = 0; t < rin; ++t) {
                double z = zrow[t];
                const double* krow = K + t * cols;
                for (int64_t q = 0; q < cols; ++q) brow[q] += z * krow[q];
            }
        }
        rows *= dims[l];
        if (l != d - 1) { double* tmp = za; za = zb; zb = tmp; }
    }
    free(za);
    free(zb);
    return 0;
}

/* One entry by the slice product G_1(i_1) G_2(i_2) ... G_d(i_d) (Sec. 5.1),
 * left to right: the independent core-chain evaluator of Sec. 3.4. */
double orc_tt_entry(const double* const* cores, const int64_t* dims, const int64_t* ranks,
                    int d, const int64_t* idx)
{
    int64_t rmax = 1;
    for (int l = 0; l <= d; ++l) if (ranks[l] > rmax) rmax = ranks[l];
    double* v = (double*)calloc((size_t)rmax, sizeof(double));
    double* w = (double*)calloc((size_t)rmax, sizeof(double));
    int64_t r1 = ranks[1];
    for (int64_t t = 0; t < r1; ++t) v[t] = cores[0][idx[0] * r1 + t];
    for (int l = 1; l < d; ++l) {
        int64_t ra = ranks[l], rb = ranks[l + 1], nl = dims[l];
        const double* G = cores[l];
        for (int64_t q = 0; q < rb; ++q) {
            double acc = 0.0;
            for (int64_t t = 0; t < ra; ++t) acc += v[t] * G[(t * nl + idx[l]) * rb + q];
            w[q] = acc;
        }
        double* tmp = v; v = w; w = tmp;
    }
    double res = v[0];
    free(v);
    free(w);
    return res;
}

/* ------------------------------------------------------------------------ */
/* Sums of squares (Frobenius norm, Sec. 5.1).  Kahan-compensated, ascending.*/
/* ------------------------------------------------------------------------ */
double orc_sumsq(const double* a, int64_t n)
{
    double s = 0.0, c = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        double y = a[i] * a[i] - c;
        double t = s + y;
        c = (t - s) - y;
        s = t;
    }
    return s;
}

double orc_sumsq_diff(const double* a, const double* b, int64_t n)
{
    double s = 0.0, c = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        double d = a[i] - b[i];
        double y = d * d - c;
        double t = s + y;
        c = (t - s) - y;
        s = t;
    }
    return s;
}

/* ------------------------------------------------------------------------ */
/* Householder QR (Golub & Van Loan, Alg. 5.2.1), thin form.                 */
/* A is m x n row-major with m >= n.  On return Q (m x n, row-major) has     */
/* orthonormal columns and R (n x n, row-major) is upper triangular with     */
/* diag(R) >= 0, which makes the factorization unique for full-rank A.       */
/* ------------------------------------------------------------------------ */
int orc_qr(const double* A, int64_t m, int64_t n, double* Q, double* R)
{
    if (m < n || n < 0) return -1;
    if (n == 0) return 0;
    /* work in column-major so Householder vectors and columns are contiguous */
    double* W = (double*)malloc((size_t)(m * n) * sizeof(double));
    double* beta = (double*)calloc((size_t)n, sizeof(double));
    if (!W || !beta) { free(W); free(beta); return -2; }
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j) W[j * m + i] = A[i * n + j];

    /* Householder vectors v_j are stored below the diagonal of W with the
     * leading entry kept in vlead[j]; R is stored on and above the diagonal. */
    double* vlead = (double*)calloc((size_t)n, sizeof(double));
    for (int64_t j = 0; j < n; ++j) {
        double* x = W + j * m;                 /* column j, rows j..m-1 */
        double norm2 = 0.0;
        for (int64_t i = j; i < m; ++i) norm2 += x[i] * x[i];
        double nrm = sqrt(norm2);
        if (nrm == 0.0) { beta[j] = 0.0; vlead[j] = 0.0; continue; }
        double alpha = (x[j] >= 0.0) ? -nrm : nrm;   /* x -> alpha e_1 */
        double v0 = x[j] - alpha;
        /* v = [v0, x[j+1..]], beta = 2 / (v^T v) */
        double vtv = v0 * v0;
        for (int64_t i = j + 1; i < m; ++i) vtv += x[i] * x[i];
        beta[j] = (vtv > 0.0) ? 2.0 / vtv : 0.0;
        vlead[j] = v0;
        x[j] = alpha;
        /* apply H_j = I - beta v v^T to the trailing columns */
        #pragma omp parallel for schedule(static)
        for (int64_t c = j + 1; c < n; ++c) {
            double* y = W + c * m;
            double dot = v0 * y[j];
            for (int64_t i = j + 1; i < m; ++i) dot += x[i] * y[i];
            double f = beta[j] * dot;
            y[j] -= f * v0;
            for (int64_t i = j + 1; i < m; ++i) y[i] -= f * x[i];
        }
    }
    /* R */
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < n; ++j) R[i * n + j] = (j >= i) ? W[j * m + i] : 0.0;
    /* Q = H_0 H_1 ... H_{n-1} [I_n; 0], accumulated backwards, column-major */
    double* Qc = (double*)calloc((size_t)(m * n), sizeof(double));
    for (int64_t j = 0; j < n; ++j) Qc[j * m + j] = 1.0;
    for (int64_t j = n - 1; j >= 0; --j) {
        const double* x = W + j * m;
        double v0 = vlead[j];
        if (beta[j] == 0.0) continue;
        #pragma omp parallel for schedule(static)
        for (int64_t c = 0; c < n; ++c) {
            double* y = Qc + c * m;
            double dot = v0 * y[j];
            for (int64_t i = j + 1; i < m; ++i) dot += x[i] * y[i];
            double f = beta[j] * dot;
            y[j] -= f * v0;
            for (int64_t i = j + 1; i < m; ++i) y[i] -= f * x[i];
        }
    }
    /* sign convention diag(R) >= 0 */
    for (int64_t j = 0; j < n; ++j) {
        if (R[j * n + j] < 0.0) {
            for (int64_t c = j; c < n; ++c) R[j * n + c] = -R[j * n + c];
            for (int64_t i = 0; i < m; ++i) Qc[j * m + i] = -Qc[j * m + i];
        }
    }
    for (int64_t i = 0; i < m; ++i)
        for (int64_t j = 0; j < n; ++j) Q[i * n + j] = Qc[j * m + i];
    free(Qc);
    free(vlead);
    free(W);
    free(beta);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* One-sided Jacobi SVD (Hestenes; Demmel & Veselic) of a square n x n      */
/* matrix B (row-major): B = U diag(S) V^T.  Column pairs (p, q) are         */
/* rotated, cyclic by rows, until every pair is orthogonal to working        */
/* precision.  S is sorted non-increasing; the largest-magnitude entry of    */
/* every left singular vector is made positive.  Returns the sweep count,    */
/* or a negative value if it did not converge.                               */
/* ------------------------------------------------------------------------ */
int orc_jacobi_svd(const double* B, int64_t n, double* U, double* S, double* V)
{
    if (n <= 0) return 0;
    double* W = (double*)malloc((size_t)(n * n) * sizeof(double));   /* columns of B */
    double* Vc = (double*)calloc((size_t)(n * n), sizeof(double));   /* columns of V */
    if (!W || !Vc) { free(W); free(Vc); return -2; }
    for (int64_t i = 0; i < n; ++i)
        for (int64_t j = 0; j < n; ++j) W[j * n + i] = B[i * n + j];
    for (int64_t j = 0; j < n; ++j) Vc[j * n + j] = 1.0;

    /* a computed inner product of two orthogonal columns carries rounding
     * noise of order n * eps * |w_p| |w_q|, so that is the smallest
     * threshold every pair can reach */
    const double tol = (n > 4 ? (double)n : 4.0) * 2.220446049250313e-16;
    int sweep, converged = 0;
    for (sweep = 1; sweep <= 80; ++sweep) {
        int64_t rotations = 0;
        for (int64_t p = 0; p < n - 1; ++p) {
            for (int64_t q = p + 1; q < n; ++q) {
                double* wp = W + p * n;
                double* wq = W + q * n;
                double alpha = 0.0, beta = 0.0, gamma = 0.0;
                for (int64_t i = 0; i < n; ++i) {
                    alpha += wp[i] * wp[i];
                    beta += wq[i] * wq[i];
                    gamma += wp[i] * wq[i];
                }
                /* a column whose squared norm is below the smallest normal
                 * number is numerically zero; sqrt(alpha) sqrt(beta) (not
                 * sqrt(alpha beta)) keeps the test free of underflow */
                if (alpha < 2.2250738585072014e-308 || beta < 2.2250738585072014e-308) continue;
                if (gamma == 0.0 || fabs(gamma) <= tol * sqrt(alpha) * sqrt(beta)) continue;
                ++rotations;
                double zeta = (beta - alpha) / (2.0 * gamma);
                double t = (zeta >= 0.0 ? 1.0 : -1.0) / (fabs(zeta) + hypot(1.0, zeta));
                double c = 1.0 / sqrt(1.0 + t * t);
                double s = c * t;
                for (int64_t i = 0; i < n; ++i) {
                    double a = wp[i], b = wq[i];
                    wp[i] = c * a - s * b;
                    wq[i] = s * a + c * b;
                }
                double* vp = Vc + p * n;
                double* vq = Vc + q * n;
                for (int64_t i = 0; i < n; ++i) {
                    double a = vp[i], b = vq[i];
                    vp[i] = c * a - s * b;
                    vq[i] = s * a + c * b;
                }
            }
        }
        if (rotations == 0) { converged = 1; break; }
    }
    /* singular values = column norms; order non-increasing (stable) */
    double* nrm = (double*)malloc((size_t)n * sizeof(double));
    int64_t* order = (int64_t*)malloc((size_t)n * sizeof(int64_t));
    for (int64_t j = 0; j < n; ++j) {
        double s2 = 0.0;
        for (int64_t i = 0; i < n; ++i) s2 += W[j * n + i] * W[j * n + i];
        nrm[j] = sqrt(s2);
        order[j] = j;
    }
    for (int64_t a = 1; a < n; ++a) {          /* insertion sort, stable */
        int64_t key = order[a];
        int64_t b = a - 1;
        while (b >= 0 && nrm[order[b]] < nrm[key]) { order[b + 1] = order[b]; --b; }
        order[b + 1] = key;
    }
    for (int64_t jj = 0; jj < n; ++jj) {
        int64_t j = order[jj];
        double sv = nrm[j];
        S[jj] = sv;
        double* w = W + j * n;
        double* v = Vc + j * n;
        /* left vector: w / sv; a zero column gets e_jj (any unit vector
         * completes the factorization) */
        double big = 0.0;
        int64_t bigi = 0;
        for (int64_t i = 0; i < n; ++i) {
            double ui = (sv > 0.0) ? w[i] / sv : (i == jj ? 1.0 : 0.0);
            U[i * n + jj] = ui;
            if (fabs(ui) > big) { big = fabs(ui); bigi = i; }
        }
        double sg = (U[bigi * n + jj] < 0.0) ? -1.0 : 1.0;
        for (int64_t i = 0; i < n; ++i) {
            U[i * n + jj] *= sg;
            V[i * n + jj] = sg * v[i];
        }
    }
    free(nrm);
    free(order);
    free(W);
    free(Vc);
    return converged ? sweep : -1;
}

/* Product C = A B for A (m x p) and B (p x n), row-major, ascending sums.
 * Used to combine the QR and Jacobi factors of a rectangular SVD. */
void orc_matmul(const double* A, const double* B, double* C, int64_t m, int64_t p, int64_t n)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double* crow = C + i * n;
        for (int64_t j = 0; j < n; ++j) crow[j] = 0.0;
        for (int64_t t = 0; t < p; ++t) {
            double a = A[i * p + t];
            const double* brow = B + t * n;
            for (int64_t j = 0; j < n; ++j) crow[j] += a * brow[j];
        }
    }
}

/* Thread count of later parallel loops (timing of the one-thread baseline);
 * results do not depend on it (every loop's sums run in a fixed order). */
void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    omp_set_num_threads(n > 0 ? n : 1);
#else
    (void)n;
#endif
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

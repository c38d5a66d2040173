/*
 * lrc.h -- C ABI of the low-precision rank-compensation hot path on AMD
 * Instinct MI355X (gfx950).
 *
 * Problem statements follow El Mountasser & Jbilou, "Low-Precision Rank
 * Compensation for Matrices and Tensor Trains":
 *   - factor apply, Sec. 4.4 eq. gpu_matrix_apply;
 *   - Tensor-Train reconstruction, Sec. 5.1 and Sec. 7.5
 *     eq. gpu_tt_reconstruction;
 *   - certificates, Thm thm:matrix_rank_compensation (Sec. 4.1) and
 *     Thm thm:tt_conditional (Sec. 6) with Algorithm alg:tt_compensation
 *     (Sec. 7.1);
 *   - storage counts, Sec. 4.2 and Sec. 5.1.
 *
 * Conventions shared by every entry point
 *   Pointers.  Arrays named "device" live in device memory of the current
 *     HIP device (hipSetDevice / torch.cuda.set_device).  Arrays named
 *     "host" live in host memory.  The caller owns every array; the library
 *     never frees, reallocates or writes a caller input.
 *   Layout.  Dense, row-major (C order), no padding, every element in the
 *     storage precision `prec` unless stated otherwise.
 *   Precision codes.  LRC_FP64 = IEEE binary64 with binary64 accumulation;
 *     LRC_FP32 = binary32 with binary32 accumulation; LRC_FP16 = binary16
 *     storage with binary32 accumulation (the paper's protocol, Sec. 3.4).
 *   Streams.  Work is enqueued on the calling thread's stream
 *     (lrc_set_stream, default the null stream).  lrc_matrix_apply and
 *     lrc_tt_reconstruct return without synchronizing; lrc_certify
 *     synchronizes its stream before it returns.
 *   Errors.  0 on success, a negative LRC_E* code otherwise; the message is
 *     available from lrc_last_error() on the same thread.  All argument
 *     checks run on the host before any HIP call; outputs are unspecified
 *     after an error.  No C++ exception crosses this interface.
 *   Workspace.  The library keeps one grow-only device workspace per
 *     (device, stream), allocated on first use and released by
 *     lrc_shutdown().  Calls on the same stream are ordered; calls issued
 *     concurrently from several host threads on the SAME stream race on it.
 */
#ifndef LRC_H
#define LRC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LRC_VERSION 1

/* storage precisions */
#define LRC_FP64 0
#define LRC_FP32 1
#define LRC_FP16 2

/* return codes */
#define LRC_OK 0
#define LRC_EINVAL (-1)     /* null pointer, bad size, rank, precision or aliasing */
#define LRC_EOVERFLOW (-2)  /* a size or byte count overflows int64 */
#define LRC_EHIP (-3)       /* HIP runtime or launch error */
#define LRC_ENOMEM (-4)     /* device workspace allocation failed */
#define LRC_ENODEV (-5)     /* no gfx950 device is current */
#define LRC_ENUMERIC (-6)   /* a factorization met a numerically rank-deficient matrix */

/* apply kernels (regime dispatch, Sec. 4.4: the speedup depends strongly on
 * the batch size) */
#define LRC_PATH_AUTO 0     /* choose by batch size */
#define LRC_PATH_STREAM 1   /* streaming wavefront-reduction path (small batch) */
#define LRC_PATH_MFMA 2     /* matrix-core path (large batch) */

/* certificate kinds */
#define LRC_CERT_MATRIX 0
#define LRC_CERT_TT 1

/* Outcomes of Algorithm alg:tt_compensation (Sec. 7.1), also used for the
 * matrix certificate. */
#define LRC_OUTCOME_FALLBACK 0       /* keep the FP64 baseline */
#define LRC_OUTCOME_CERTIFIED 1      /* certified non-increase, no memory win */
#define LRC_OUTCOME_CERTIFIED_MEM 2  /* certified non-increase and memory win */

/*
 * lrc_matrix_apply -- Y = U diag(s) (V^T X)   (Sec. 4.4 eq. gpu_matrix_apply)
 *
 * The paper writes the product for a b x n batch X_p as
 * Y_p = [(X_p V_r) diag(s_r)] U_r^T; here X = X_p^T (n x batch) and
 * Y = Y_p^T (m x batch), so the numbers are identical.
 *   U  device, m x k      stored left factor U_k
 *   s  device, k          stored singular values s_k
 *   V  device, n x k      stored right factor V_k (V, not V^T)
 *   X  device, n x batch  input batch
 *   Y  device, m x batch  output, written in `prec`; must not overlap any input
 * Phase 1 forms T' = diag(s) V^T X in the accumulation precision (for FP16
 * it is rounded once to binary16 as the input of the second product);
 * phase 2 forms Y = U T'.  Sums are split in a fixed order, so the result is
 * bitwise reproducible run to run.
 * Errors: LRC_EINVAL if a pointer is NULL, m, n, k or batch < 1, k >
 * min(m, n), prec is unknown or Y overlaps an input; LRC_EOVERFLOW if an
 * element count overflows; LRC_ENOMEM / LRC_EHIP / LRC_ENODEV from the
 * runtime.
 */
int lrc_matrix_apply(const void* U, const void* s, const void* V, const void* X, void* Y,
                     int64_t m, int64_t n, int64_t k, int64_t batch, int prec);

/*
 * lrc_matrix_apply_noalloc -- lrc_matrix_apply without any allocation
 *
 * For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, kernels, plan and result (bit for bit) as lrc_matrix_apply;
 * the split sums and T' live in a fixed scratch array of
 * LRC_NOALLOC_SCRATCH_BYTES in device memory instead of the library's
 * grow-only workspace.  Each device holds its own array from the first call
 * until the process ends; no hipMalloc, hipFree or allocating library
 * routine is called (with kernel timing off, the default).
 * Every call on one device shares that device's array and leaves its last
 * contents there: calls that overlap in time on one device (two streams,
 * two threads) race on it and must be serialized by the caller.
 * Errors: those of lrc_matrix_apply, and LRC_EINVAL when the plan for these
 * sizes needs more than LRC_NOALLOC_SCRATCH_BYTES of scratch (checked on
 * the host before anything is launched).
 */
#define LRC_NOALLOC_SCRATCH_BYTES (64LL << 20)
int lrc_matrix_apply_noalloc(const void* U, const void* s, const void* V, const void* X, void* Y,
                             int64_t m, int64_t n, int64_t k, int64_t batch, int prec);

/* The apply kernel pair LRC_PATH_AUTO selects for these sizes (pure host
 * function, no device needed).  Returns LRC_PATH_STREAM or LRC_PATH_MFMA, or
 * LRC_EINVAL for invalid sizes. */
int lrc_matrix_apply_path(int64_t m, int64_t n, int64_t k, int64_t batch, int prec);

/* Force the apply kernel pair used by later lrc_matrix_apply calls on the
 * calling thread (LRC_PATH_AUTO restores the dispatch).  Returns LRC_EINVAL
 * for an unknown path. */
int lrc_set_apply_path(int path);

/*
 * lrc_tt_reconstruct -- dense tensor from Tensor-Train cores
 *   T(i_1..i_d) = G_1(i_1) G_2(i_2) ... G_d(i_d)   (Sec. 5.1; Sec. 7.5)
 *   cores  host array of d device pointers; core l (0-based) is
 *          ranks[l] x dims[l] x ranks[l+1], row-major, in `prec`
 *   dims   host, d mode sizes n_l >= 1
 *   ranks  host, d+1 TT ranks with ranks[0] = ranks[d] = 1, all >= 1
 *   d      number of cores, 1 <= d <= LRC_TT_MAX_D
 *   out    device, prod(dims) entries in C order (i_d fastest), in `prec`;
 *          must not overlap a core
 * The cores are contracted left to right (the paper's reshape chain) with
 * the partial interfaces kept on chip and the last contraction fused with
 * the output stores; intermediate sums use the accumulation precision and,
 * for FP16, the last interface is rounded once to binary16.
 * On-chip limits.  Every rank up to LRC_TT_MAX_RANK is accepted for d <= 3
 * in every precision, and for d >= 4 in FP32 and FP16.  FP64 trains of four
 * or more cores whose last rank r_{d-1} exceeds 68 keep, per workgroup, 16
 * rows of Z_{d-2} and Z_{d-1} plus two chain rows of the left interface in
 * LDS: 128 (r_{d-2} + r_{d-1}) + 16 B max(r_1 .. r_{d-2}) bytes (B = 16,
 * or 16 / n_{d-1} rounded down when n_{d-1} < 16), which must fit the
 * device's 160 KB (about rank 300 with B = 16 and equal ranks); larger ones
 * return LRC_EINVAL.
 * Errors: LRC_EINVAL for NULL pointers, d out of range, a dimension or rank
 * < 1, ranks[0] or ranks[d] != 1, a rank above LRC_TT_MAX_RANK or beyond the
 * on-chip limits above, an unknown prec or overlapping output;
 * LRC_EOVERFLOW if prod(dims) overflows.
 */
#define LRC_TT_MAX_D 16
#define LRC_TT_MAX_RANK 512
int lrc_tt_reconstruct(const void* const* cores, const int64_t* dims, const int64_t* ranks,
                       int d, void* out, int prec);

/*
 * lrc_certify -- rank-compensation certificate
 *
 * Matrix (kind = LRC_CERT_MATRIX), Thm thm:matrix_rank_compensation:
 *   base rank k in FP64, compensated rank k+1 stored in `prec`.
 *   sigma       host, all n_sigma = min(m, n) singular values of A,
 *               non-increasing (the tails E_k, E_{k+1} sum over the whole
 *               spectrum; a truncated spectrum is rejected)
 *   U, s, V     device FP64 rank-(k+1) factors: U m x (k+1), s (k+1), V n x (k+1)
 *   Uh, sh, Vh  device, the same factors as stored in `prec` (each rounded
 *               individually, Remark after the theorem)
 *   A           device FP64 m x n, or NULL (then err_new is NaN and the
 *               accuracy-win flags are 0)
 *   E_k and E_{k+1} come from sigma (Eckart-Young); eta = ||A_{k+1} -
 *   A_hat_{k+1}||_F with both contracted in FP64; certified iff
 *   E_{k+1} + eta <= E_k, compared exactly in FP64 (eq. matrix_condition).
 *
 * Tensor Train (kind = LRC_CERT_TT), Thm thm:tt_conditional, Algorithm
 * alg:tt_compensation steps 5-9:
 *   d, dims     host, as in lrc_tt_reconstruct
 *   T           device FP64 dense tensor (C order), required
 *   ranks_base, cores_base   host ranks / host array of device FP64 cores
 *                            of the baseline T_R
 *   ranks_aug, cores_aug     the same for the augmented FP64 T_{R+}, in the
 *                            gauge that was rounded (left-orthogonal)
 *   cores_aug_h              host array of device cores of T_{R+} as
 *                            stored in `prec`
 *   E_R = ||T - T_R||, E_{R+} = ||T - T_{R+}||, S_TT = E_R^2 - E_{R+}^2,
 *   eta_TT = ||T_{R+} - T_hat_{R+}||, all contracted in FP64; certified iff
 *   E_{R+} + eta_TT <= E_R (eq. tt_condition).
 *
 * Result fields: absolute Frobenius values (divide by norm_ref for the
 * paper's relative units); bytes are exact stored bytes (Sec. 4.2 / 5.1);
 * the flags follow the vocabulary of Sec. 4.1 with strict comparisons for
 * wins.  Synchronizes the stream.
 * Errors: LRC_EINVAL for missing arrays, inconsistent sizes or ranks, prec
 * not FP32/FP16/FP64, n_sigma != min(m, n), or sigma not non-increasing.
 */
typedef struct lrc_cert_args {
    int kind;                       /* LRC_CERT_MATRIX or LRC_CERT_TT */
    int prec;                       /* storage precision of the compensated form */
    /* matrix */
    int64_t m, n, k;
    const double* sigma;            /* host */
    int64_t n_sigma;
    const double* U;                /* device FP64 */
    const double* s;
    const double* V;
    const void* Uh;                 /* device, prec */
    const void* sh;
    const void* Vh;
    const double* A;                /* device FP64 or NULL */
    /* tensor train */
    int d;
    const int64_t* dims;            /* host */
    const double* T;                /* device FP64 */
    const int64_t* ranks_base;      /* host, d+1 */
    const double* const* cores_base;    /* host array of device pointers */
    const int64_t* ranks_aug;       /* host, d+1 */
    const double* const* cores_aug;     /* host array of device pointers */
    const void* const* cores_aug_h;     /* host array of device pointers, prec */
} lrc_cert_args;

typedef struct lrc_cert_result {
    double E_base;       /* E_k or E_R */
    double E_aug;        /* E_{k+1} or E_{R+} */
    double eta;          /* eta_{k+1} or eta_TT */
    double err_new;      /* ||A - A_hat|| or ||T - T_hat|| (NaN if A is NULL) */
    double gain;         /* sigma_{k+1}^2 or S_TT */
    double margin;       /* E_base - E_aug - eta */
    double norm_ref;     /* ||A||_F (from sigma) or ||T||_F */
    int64_t bytes_base;  /* FP64 storage at the base rank */
    int64_t bytes_aug;   /* `prec` storage at the compensated rank */
    int certified;       /* E_aug + eta <= E_base */
    int acc_nonincrease; /* err_new <= E_base */
    int acc_win;         /* err_new <  E_base */
    int mem_win;         /* bytes_aug < bytes_base */
    int practical_win;   /* acc_win && mem_win */
    int outcome;         /* LRC_OUTCOME_* */
} lrc_cert_result;

int lrc_certify(const lrc_cert_args* args, lrc_cert_result* res);

/*
 * lrc_round -- stored values from binary64 values: y[i] = round(x[i])
 * (Sec. 3.2 formats; Remark after Thm thm:matrix_rank_compensation: every
 * factor entry is rounded on its own; Algorithm alg:tt_compensation,
 * rounding step for the TT cores)
 *   x           device, count binary64 values
 *   y           device, count values in `prec`; must not overlap x
 *   count       >= 0 (0: nothing is launched; x and y may then be NULL)
 *   prec        LRC_FP32 or LRC_FP16 (LRC_FP64 copies x)
 *   n_overflow  host, or NULL.  When given, the call waits for the result
 *               and stores the number of finite inputs that rounded to
 *               +-infinity.
 * One round-to-nearest-even step from binary64 (never through binary32 on
 * the way to binary16); subnormal results are kept; finite values from the
 * midpoint above the largest finite value up become +-infinity; +-infinity
 * stays; NaN becomes the quiet NaN of the same sign (payload not kept).
 * Enqueued on the calling thread's stream; without n_overflow it returns
 * without synchronizing.
 * Errors: LRC_EINVAL for NULL x or y with count > 0, count < 0, an unknown
 * prec or y overlapping x; LRC_EOVERFLOW if 8 count overflows; LRC_EHIP /
 * LRC_ENODEV from the runtime.
 */
int lrc_round(const void* x, void* y, int64_t count, int prec, int64_t* n_overflow);

/*
 * lrc_tt_left_orthogonalize -- left-orthogonal gauge of FP64 TT cores, in
 * place (Sec. 6.1; Algorithm alg:tt_compensation, gauge step)
 *   For l = 1..d-1 the left unfolding of core l, A_l of size
 *   (r_{l-1} n_l) x r_l, is factored A_l = Q_l R_l with Q_l^T Q_l = I and
 *   diag(R_l) > 0; core l becomes Q_l and the left unfolding of core l+1
 *   (r_l x n_{l+1} r_{l+1}) is replaced by R_l times itself.  The tensor
 *   the train represents is unchanged up to rounding.
 *   cores  host array of d device pointers to binary64 cores (ranks[l] x
 *          dims[l] x ranks[l+1], row-major), overwritten; no two overlap
 *   dims, ranks, d  as for lrc_tt_reconstruct, with ranks[l] <=
 *          LRC_GAUGE_MAX_RANK and ranks[l-1] dims[l-1] >= ranks[l] for
 *          1 <= l <= d-1
 * Each QR is computed as CholeskyQR2 (two passes of: Gram matrix on the
 * FP64 matrix cores, Cholesky, triangular right product), which with
 * positive diagonals gives the same factors as a Householder QR up to
 * rounding while the unfolding's condition number stays below about 1e7.
 * Synchronizes the calling thread's stream before it returns.
 * Errors: LRC_EINVAL for NULL pointers, an invalid shape, a rank above
 * LRC_GAUGE_MAX_RANK, an unfolding with fewer rows than columns or
 * overlapping cores; LRC_ENUMERIC when an unfolding is numerically rank
 * deficient for this method (a Cholesky pivot at or below 2^-46 of its
 * column's squared norm; the cores are then unspecified); LRC_EOVERFLOW,
 * LRC_ENOMEM, LRC_EHIP, LRC_ENODEV as elsewhere.
 */
#define LRC_GAUGE_MAX_RANK 96
int lrc_tt_left_orthogonalize(void* const* cores, const int64_t* dims, const int64_t* ranks, int d);

/*
 * Fixed-memory comparison tools (Sec. sec:hyperspectral_application).
 *
 * Quality of a reconstruction Xh against its FP64 reference X, both with
 * the spectral bands as the last (contiguous) mode:
 *   rel_err     ||X - Xh||_F / ||X||_F
 *   psnr        mean over bands b of 20 log10(L_b / sqrt(MSE_b)), L_b the
 *               band's range (max(max|X_b|, 1) for a constant band);
 *               +infinity when a band is reproduced exactly
 *   ssim        mean over bands of the SSIM variant evaluated once per whole
 *               band with population means, variances and covariance,
 *               C1 = (0.01 L_b)^2, C2 = (0.03 L_b)^2
 *   sam         mean spectral angle (radians) over the sam_pixels pixels
 *               whose reference and reconstructed spectra both have
 *               positive norm (NaN if there are none)
 * Sums are added in a fixed order: results are bitwise reproducible.
 */
typedef struct {
    double rel_err, psnr, ssim, sam;
    int64_t sam_pixels;
    int64_t pixels, bands;
} lrc_quality;

/* Dense pair: X device FP64 and Xh device in `prec`, both pixels x bands
 * row-major; Xh is multiplied by `scale` as it is read (1.0: as stored;
 * the norm of a normalized tensor undoes the normalization).  Synchronizes
 * the calling thread's stream.  Errors: LRC_EINVAL (NULL pointer, pixels or
 * bands < 1, unknown prec), LRC_EOVERFLOW, LRC_ENOMEM, LRC_EHIP, LRC_ENODEV. */
int lrc_band_quality(const void* X, const void* Xh, int64_t pixels, int64_t bands, int prec, double scale,
                     lrc_quality* q);

/* TT cores (as for lrc_tt_reconstruct, stored in `prec`, d >= 2) against the
 * device FP64 reference X (Sec. sec:hyperspectral_application): the stored
 * cores are widened exactly and contracted in FP64 (the paper's evaluation
 * of rounded cores), the result multiplied by `scale`, and measured as
 * lrc_band_quality does, with bands = dims[d-1] and pixels = the product of
 * the other modes.  When the FP64 reconstruction runs by wave tiles (d >= 3,
 * last rank <= 68, at most 455 bands) the measures are formed in its
 * epilogue, which reads only the cores and X; otherwise the dense FP64
 * reconstruction is written to the library's workspace and measured in two
 * passes.  Sums are added in a fixed order either way (bitwise reproducible
 * for a given path).  Synchronizes.  Errors as lrc_tt_reconstruct, plus
 * LRC_EINVAL for d < 2 or a NULL X. */
int lrc_tt_quality(const void* const* cores, const int64_t* dims, const int64_t* ranks, int d, int prec,
                   const void* X, double scale, lrc_quality* q);

/* Memory-matched FP64 rank: the largest uniform nominal TT rank R whose
 * exact FP64 storage (8 sum_l r_{l-1} n_l r_l, ranks capped by the
 * unfolding dimensions, r_l <= min(R, r_{l-1} n_l, prod_{i>l} n_i)) does
 * not exceed budget_bytes.  Writes the d+1 capped ranks to ranks_out (host)
 * and returns R, or returns 0 (ranks_out all 0) if rank 1 does not fit.
 * Pure host function.  Errors: LRC_EINVAL for NULL pointers, d outside
 * [1, LRC_TT_MAX_D] or a dimension < 1. */
int64_t lrc_tt_memory_matched_rank(const int64_t* dims, int d, int64_t budget_bytes, int64_t* ranks_out);

/* ---- Randomized FP64 factorization (the end-to-end decomposition left to
 * future work in Sec. sec:conclusion): the randomized range finder of
 * Halko, Martinsson and Tropp (2011) with an exact SVD of the projected
 * matrix, and TT-SVD (Sec. 5.1, eq. tt_svd_error) built on it.  The test
 * vectors are drawn by the caller (Gaussian in the intended use). */
#define LRC_RSVD_MAX_SAMPLES 96
#define LRC_RSVD_MAX_POWER_ITERS 8

/* Rank-k randomized SVD of the device FP64 matrix A (m x n, row-major) with
 * the l test vectors given as the rows of omega (l x n, device FP64):
 *   Y = A omega^T, Q = orth(Y); power_iters times Q = orth(A orth(A^T Q));
 *   B = Q^T A = Ub diag(s) Vt (exact SVD of the small matrix);
 *   U = Q Ub[:, :k], V = Vt[:k]^T,
 * so that U diag(s) V^T = U U^T A.  Outputs (device, FP64, written whole):
 * U (m x k), s (k, non-increasing), V (n x k), all row-major.  The factors
 * are unique up to the sign of each singular pair when the singular values
 * are distinct; a singular value that is exactly zero gets a zero column in
 * U.  Orthonormalizations are CholeskyQR2 (as lrc_tt_left_orthogonalize);
 * when one breaks down (condition number above about 1e7) the whole call is
 * repeated once with shifted CholeskyQR3, which holds to about 1e15; the
 * small SVD is one-sided Jacobi.  Synchronizes the calling thread's stream.
 * Errors: LRC_EINVAL (NULL pointer, sizes outside 1 <= k <= l <= min(m, n),
 * l > LRC_RSVD_MAX_SAMPLES, power_iters outside [0,
 * LRC_RSVD_MAX_POWER_ITERS], an output overlapping an input or another
 * output), LRC_ENUMERIC (a sketch or projected matrix numerically rank
 * deficient even for shifted CholeskyQR3, e.g. a matrix of rank below l, or
 * a Jacobi sweep limit reached), LRC_EOVERFLOW, LRC_ENOMEM, LRC_EHIP,
 * LRC_ENODEV. */
int lrc_rsvd(const double* A, int64_t m, int64_t n, const double* omega, int64_t l, int power_iters, int64_t k,
             double* U, double* s, double* V);

/* Randomized TT-SVD of the device FP64 tensor T (dims[0..d-1], C order,
 * d >= 2): step l = 0..d-2 factors C_l ((ranks[l] dims[l]) x prod_{i>l}
 * dims[i], C_0 = T) as lrc_rsvd does with samples[l] test vectors
 * omegas[l] (samples[l] x prod_{i>l} dims[i], device FP64) at rank
 * ranks[l+1]; core l = U (ranks[l] x dims[l] x ranks[l+1]) and C_{l+1} =
 * diag(s) V^T, whose last value is the last core.  ranks has d+1 entries
 * with ranks[0] = ranks[d] = 1 and 1 <= ranks[l+1] <= samples[l] <= both
 * sizes of C_l, samples[l] <= LRC_RSVD_MAX_SAMPLES.  cores: d device FP64
 * buffers (written whole).  sigma (device, may be NULL): the kept singular
 * values of every step, concatenated (sum of ranks[1..d-1] values).
 * Synchronizes.  Errors as lrc_rsvd (LRC_ENUMERIC names the step). */
int lrc_tt_rsvd(const double* T, const int64_t* dims, const int64_t* ranks, int d, const double* const* omegas,
                const int64_t* samples, int power_iters, double* const* cores, double* sigma);

/* Stored bytes of rank-k factors in `prec`: (b/8) k (m+n+1)  (Sec. 4.2).
 * Returns LRC_EINVAL for bad arguments or LRC_EOVERFLOW on overflow. */
int64_t lrc_storage_bytes(int64_t m, int64_t n, int64_t k, int prec);

/* Stored bytes of TT cores: (b/8) sum_l R_{l-1} n_l R_l  (Sec. 5.1).
 * dims and ranks are host arrays of length d and d+1. */
int64_t lrc_tt_storage_bytes(const int64_t* dims, const int64_t* ranks, int d, int prec);

/* Stream for later calls on the calling thread (a hipStream_t; NULL = the
 * null stream).  Never fails. */
int lrc_set_stream(void* hip_stream);

/* Message for the last non-zero return on the calling thread ("" if none).
 * The pointer stays valid until the next call on the same thread. */
const char* lrc_last_error(void);

/* Releases every library-owned device workspace.  Later calls allocate
 * again.  No call may be in flight. */
void lrc_shutdown(void);

/*
 * Kernel timing (measurement tools).  While enabled, the library records a
 * pair of hipEvents on the launch stream around every kernel it launches,
 * labelled by kernel ("apply_p2_mfma_f16", "tt_fused_f64", ...); the extra
 * event records cost a few microseconds per launch.  lrc_profile_read
 * waits for the recorded events and returns the number of launches and the
 * summed elapsed milliseconds for one label (0 and 0.0 if unseen).
 * lrc_profile_labels writes the comma-separated labels seen so far into buf
 * (truncated to len-1 characters) and returns the full length.
 */
int lrc_profile_enable(int on);
/* Restricts the event pairs to launches whose label equals `label` (NULL or
 * "" removes the restriction), so that one kernel can be timed inside a
 * longer run at the cost of its own two event records only. */
int lrc_profile_filter(const char* label);
void lrc_profile_reset(void);
int lrc_profile_read(const char* label, int64_t* launches, double* total_ms);
int64_t lrc_profile_labels(char* buf, int64_t len);

/* LRC_VERSION of the built library. */
int lrc_version(void);

/* Measurement aid: the matrix-core ceiling of this device, in TFLOP/s, for
 * the MFMA instruction the kernels use in `prec` (FP64 and FP32 16x16x4,
 * FP16 16x16x32 with FP32 accumulation), measured by a register-only loop of
 * independent products on every compute unit (about 10 ms, best of two
 * timed runs after a warm-up run), so that roofline fractions can be given
 * against measured as well as published peaks.  Synchronizes the calling
 * thread's stream.  Errors: LRC_EINVAL (NULL, unknown prec), LRC_ENODEV,
 * LRC_ENOMEM, LRC_EHIP. */
int lrc_mfma_ceiling(int prec, double* tflops);

#ifdef __cplusplus
}
#endif

#endif /* LRC_H */

// Host-side interface between the C ABI layer (lrc_api.cpp) and the kernel
// translation units.  Launchers validate nothing: lrc_api.cpp checks every
// argument before calling them.  Each launcher returns hipSuccess or the
// first launch error.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace lrc {

enum Prec { P64 = 0, P32 = 1, P16 = 2 };

inline int elem_bytes(int prec) { return prec == P64 ? 8 : (prec == P32 ? 4 : 2); }
inline int mfma_kb(int prec) { return prec == P16 ? 32 : 4; }
inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Grow-only device workspace; `take` hands out 256-byte aligned slices of
// one allocation, in call order, and fails with hipErrorOutOfMemory if the
// reservation made by `reserve` is exceeded.
struct Workspace {
    char* base = nullptr;
    size_t cap = 0;
    size_t used = 0;
    bool overrun = false;         // a take() exceeded the reservation
    hipError_t reserve(size_t bytes, hipStream_t stream);
    void* take(size_t bytes);     // nullptr (and overrun = true) past the reservation
    void reset() { used = 0; overrun = false; }
    void release();
};

// Kernel timing: when enabled (lrc_profile_enable), a pair of hipEvents is
// recorded on the launch stream around every kernel the library launches,
// keyed by a kernel label; lrc_profile_read sums the elapsed times.
struct KernelTimer {
    KernelTimer(const char* label, hipStream_t stream);
    ~KernelTimer();
    KernelTimer(const KernelTimer&) = delete;
    KernelTimer& operator=(const KernelTimer&) = delete;
    const char* label;
    hipStream_t stream;
    void* start;   // hipEvent_t, or nullptr when profiling is off
};

// ---------------------------------------------------------------- apply ---
struct ApplyPlan {
    int path;            // LRC_PATH_STREAM or LRC_PATH_MFMA
    int64_t Kp;          // pitch of the rows of T'^T and of staged copies of U, V (k rounded up)
    // phase 1 (split over n)
    int splits;
    int64_t chunk;       // rows of V / X per split
    int tiles_m, tiles_n;
    int big1, big2;      // 128 x 128 tiles (else 64 x 64) for phase 1 / phase 2
    // MFMA path, operands whose base or pitch rules out aligned 16-byte moves
    // (odd ranks such as the compensated k + 1, odd batches): V (phase 1,
    // mis1) and U (phase 2, mis2) are read in place when they are small or
    // read by a single tile of the other dimension; otherwise U, V (pitch Kp)
    // and X (pitch ldx) are copied to a padded pitch first
    int mis1, mis2;
    int stage_u, stage_v, stage_x;
    int64_t ldx;
    size_t stage_bytes;
    size_t part_bytes;   // partial-sum buffer
    size_t mid_bytes;    // T'^T buffer
};

// U, V, X are only inspected for alignment (may be null).
ApplyPlan plan_apply(int64_t m, int64_t n, int64_t k, int64_t b, int prec, int path, const void* U = nullptr,
                     const void* V = nullptr, const void* X = nullptr);
size_t apply_workspace_bytes(const ApplyPlan& p);

hipError_t launch_apply(const ApplyPlan& p, const void* U, const void* s, const void* V,
                        const void* X, void* Y, int64_t m, int64_t n, int64_t k, int64_t b,
                        int prec, Workspace& ws, hipStream_t stream);

// ------------------------------------------------------------ quantization
// y[i] = x[i] rounded from binary64 to prec (P32 / P16) with one
// round-to-nearest-even step; finite inputs that overflow are counted into
// *ovf (zeroed first) when ovf is not null.
hipError_t launch_round(const double* x, void* y, int64_t n, int prec, unsigned long long* ovf,
                        hipStream_t stream);

// Left-orthogonal gauge of FP64 cores in place (CholeskyQR2 per unfolding);
// flags[l] becomes 1 + pivot when the QR of unfolding l broke down.
size_t gauge_workspace_bytes(const int64_t* dims, const int64_t* ranks, int d);
hipError_t launch_gauge(double* const* cores, const int64_t* dims, const int64_t* ranks, int d, int* flags,
                        Workspace& ws, hipStream_t stream);

// Thin QR of A (rows x r inside pitch rp = r rounded to 2, 16-byte aligned,
// rows >= r) by CholeskyQR2 (the gauge's kernels), or by shifted CholeskyQR3
// when `shifted` (condition numbers up to about 1e15): Q (pitch rp, pad column
// zeroed) with Q^T Q = I and, when R is not null, R with A = Q R (rows 0..r-1
// of an rp x rp block, upper triangular, diag > 0); *flag becomes 1 + pivot
// when a Cholesky factorization breaks down (left unchanged otherwise).
size_t cholqr2_workspace_bytes(int64_t rows, int r);
hipError_t launch_cholqr2(const double* A, int64_t rows, int r, double* Q, double* R, int* flag, Workspace& ws,
                          hipStream_t stream, const char* label, bool shifted = false);
// ------------------------------------------------------ FP64 factor GEMMs ---
// out[i][j] = s_j sum_{t<K} W[j][t] A[i][t] for i < rows, j < nw (s = 1 when
// svals is null); out[i][j] = 0 for nw <= j < mout (mout <= 96 when
// nw <= 96, else at most nw rounded up to 64).  W, A: 16-byte aligned with
// even pitches.  Split-K MFMA partials summed in split order.
size_t gemm_nt_workspace_bytes(int64_t nw, int64_t rows, int64_t K);
hipError_t launch_gemm_nt(const double* W, int64_t ldw, int64_t nw, const double* A, int64_t lda, int64_t rows,
                          int64_t K, const double* svals, double* out, int64_t ldo, int64_t mout, Workspace& ws,
                          hipStream_t stream, const char* label);
// out[c][j] = sum_{i<K} Q[i][j] A[i][c] for c < cols, j < nq; zero for
// nq <= j < mout.  Same operand rules.
size_t gemm_tn_workspace_bytes(int64_t nq, int64_t cols, int64_t K);
hipError_t launch_gemm_tn(const double* Q, int64_t ldq, int64_t nq, const double* A, int64_t lda, int64_t cols,
                          int64_t K, double* out, int64_t ldo, int64_t mout, Workspace& ws, hipStream_t stream,
                          const char* label, const char* finish_label);
// ------------------------------------------------ randomized factorization
// flags: 3 ints (matrix) or 3 per step (TT), 0 on success; [0] range-finder
// QR, [1] QR of B^T, [2] Jacobi sweep limit.
size_t matrix_rsvd_workspace_bytes(int64_t m, int64_t n, int l, int k, int q);
hipError_t launch_matrix_rsvd(const double* A, int64_t m, int64_t n, const double* Om, int l, int q, int k, double* U,
                              double* s, double* V, int* flags, Workspace& ws, hipStream_t st, bool shifted = false);
size_t tt_rsvd_workspace_bytes(const int64_t* dims, const int64_t* ranks, const int64_t* samples, int d, int q);
hipError_t launch_tt_rsvd(const double* T, const int64_t* dims, const int64_t* ranks, const int64_t* samples, int d,
                          const double* const* omegas, int q, double* const* cores, double* sigma, int* flags,
                          Workspace& ws, hipStream_t st, bool shifted = false);
// ------------------------------------------------------- certificate (matrix)
// G = P^T P for P (rows x cols, row-major, FP64): a split-sum Gram product.
size_t gram_workspace_bytes(int64_t rows, int64_t cols);
hipError_t launch_gram(const double* P, int64_t rows, int64_t cols, double* G,
                       Workspace& ws, hipStream_t stream);

// P[i][t] = ref[i][t]; P[i][r + t] = widen(h[i][t]) - ref[i][t]   (rows x 2r)
hipError_t launch_diff_factors(const double* ref, const void* h, int prec, int64_t rows,
                               int64_t r, double* P, hipStream_t stream);
// W[i][t] = widen(h[i][t]) * widen(hs[t])  (hs may be NULL: factor 1), rows of
// pitch ldw >= r with zero padding
hipError_t launch_widen_scaled(const void* h, const void* hs, int prec, int64_t rows,
                               int64_t r, int64_t ldw, double* W, hipStream_t stream);
// out[i] = widen(src[i])
hipError_t launch_widen(const void* src, int prec, int64_t count, double* out, hipStream_t stream);

// --------------------------------------------------------- quality measures
// out[0..4] = relative error, mean band PSNR, mean band SSIM variant, mean
// spectral angle, pixels in that mean; X (P x B, FP64) against scale * Xh
// (P x B in prec).
// Band statistics of the quality measures, in the order of their partials:
// part[(block * QS_N + q) * B + b] (shifted sums of X and Xh, their squares
// and cross products, squared differences, squares of X, band min and max).
enum { QS_X = 0, QS_Y, QS_XX, QS_YY, QS_XY, QS_DD, QS_X2, QS_MIN, QS_MAX, QS_N };
size_t quality_workspace_bytes(int64_t P, int64_t B);
// The reductions of the band partials (nblk blocks) and the angle partials
// part2[2 k], part2[2 k + 1] (nblk2 blocks) into the five results at `out`
// (red: QS_N * B doubles of scratch).
hipError_t launch_quality_reduce(const double* part, int64_t nblk, const double* part2, int64_t nblk2,
                                 const double* X, int64_t P, int64_t B, double* red, double* out,
                                 hipStream_t stream);
hipError_t launch_quality(const double* X, const void* Xh, int prec, double scale, int64_t P, int64_t B,
                          double* out, Workspace& ws, hipStream_t stream);

// Partial sums of (A - W Vw^T)^2 over m x n, one per workgroup; returns the
// number of partials written to `part` via *nparts.
size_t err_workspace_bytes(int64_t m, int64_t n);
// part[a] for a < 2r: the per-column terms of eta^2 = trace(M^T Gu M Gq) of
// the matrix certificate (Gu, Gq: 2r x 2r Gram matrices of [U dU], [V dV]).
hipError_t launch_eta2(const double* Gu, const double* Gq, const double* s, const void* sh, int prec, int64_t r,
                       double* part, hipStream_t stream);
// W and Vw have pitch ldw (even, 16-byte aligned bases).
hipError_t launch_err_dense(const double* A, const double* W, const double* Vw, int64_t m,
                            int64_t n, int64_t r, int64_t ldw, double* part, int64_t* nparts,
                            hipStream_t stream);

// Five partial sums per workgroup over a dense tensor: (T - a)^2, (T - b)^2,
// (b - c)^2, (T - c)^2, T^2; written as part[q * groups + g].
int64_t sumsq5_groups(int64_t count);
hipError_t launch_sumsq5(const double* T, const double* a, const double* b, const double* c,
                         int64_t count, double* part, int64_t groups, hipStream_t stream);

// Fixed-order sum of `count` partials for each of `nsums` rows (part is
// nsums x count, row-major) into out[nsums] (device).
hipError_t launch_reduce_rows(const double* part, int64_t count, int nsums, double* out,
                              hipStream_t stream);

// ------------------------------------------------------------------- TT ---
constexpr int kMaxD = 16;
constexpr int kTTMaxSets = 3;

struct TTPlanSet {
    int64_t ranks[kMaxD + 1];
    int rL, rM;          // r_{d-2}, r_{d-1}
    int Kp2, Kp3;        // rL, rM rounded to the MFMA K step (Kp3: the largest over the plan's sets)
    int Rt;              // rM rounded up to 16 (row blocks of the middle product)
    int ldl, ldf;        // LDS row pitches of Z_{d-2} and Z_{d-1} (padded against bank conflicts)
};

struct TTPlan {
    int d;
    int prec;
    int nsets;           // core sets sharing one block layout (1; 3 for the certificate)
    int64_t dims[kMaxD];
    TTPlanSet set[kTTMaxSets];
    int64_t NL;          // rows of the left interface Z_{d-2} (1 when d <= 2)
    int64_t n_mid;       // n_{d-1}
    int64_t n_last;      // n_d
    // Wave tiles take a three-core train (first, middle, last).  mid is the
    // 0-based index of its middle core: d - 2, or d - 3 when the two last
    // cores are merged into one right core G_{d-1} G_d of r_{d-2} x
    // (n_{d-1} n_d) (trains with short last modes); the first core is G_1 or
    // the left interface of cores 1 .. mid.  NL, n_mid, n_last, rL and rM
    // then describe that train.
    int mid;
    int BL, BI, P;       // left rows and middle indices per block, P = BL * BI rounded to 16
    int64_t num_i_blocks, num_L_blocks;
    int grid_L;          // workgroups along the left index (each loops over L blocks)
    int chain_rmax;      // largest rank among levels 1..d-2 (chain buffers)
    size_t lds_bytes;
    size_t stage_bytes;  // staged (transposed, padded) FP16 operands
    int wave_nkb;        // FP64, d = 3 by wave tiles: K steps of the last product (0: by LDS tiles)
    int wave_npb;        // 16-row blocks per wave tile
    int64_t wave_tiles;  // wave tiles
};

// rank_sets[q] is the rank vector (d+1 entries) of core set q.  Returns 0,
// or -1 when the ranks do not fit the fused kernel's on-chip buffers
// (max_lds = the device's per-workgroup LDS limit).
// merge_right = false keeps mid = d - 2 (plans whose kernels index the last
// mode on its own, such as the fused quality measures).
int plan_tt(TTPlan& p, const int64_t* dims, const int64_t* const* rank_sets, int nsets, int d, int prec,
            size_t max_lds, bool merge_right = true);

// `label` names the launch for the kernel timers (nullptr: "tt_fused_<type>").
hipError_t launch_tt(const TTPlan& p, const void* const* cores, void* out, Workspace& ws,
                     hipStream_t stream, const char* label = nullptr);

// Fused TT certificate (FP64 plan with three core sets: base, augmented,
// widened rounded augmented): part[s * tt_cert_parts(p) + w] receives the
// five partial sums of workgroup w (order at k_tt_cert).
int64_t tt_cert_parts(const TTPlan& p);

// Matrix-core ceiling (TFLOP/s) of the kernels' MFMA instruction for `prec`
// on `cus` compute units: a register-only loop, timed with HIP events
// (synchronizes the stream).
size_t mfma_ceiling_workspace_bytes(int cus);
hipError_t launch_mfma_ceiling(int prec, int cus, double* tflops, Workspace& ws, hipStream_t st);

// Quality measures of an FP64 reconstruction (one set, wave tiles) fused
// into the reconstruction: tt_quality_blocks(p, B) is the number of
// workgroup partials the fused kernel writes (0: the plan does not take it,
// reconstruct densely instead); launch_tt_quality writes them at part
// (tt_quality_blocks * QS_N * n_d doubles) and part2 (2 per block).
int64_t tt_quality_blocks(const TTPlan& p, size_t max_lds);
hipError_t launch_tt_quality(const TTPlan& p, const void* const* cores, const double* X, double scale,
                             double* part, double* part2, size_t max_lds, Workspace& ws, hipStream_t stream);
hipError_t launch_tt_cert(const TTPlan& p, const void* const* const* cores, const double* Tref, double* part,
                          Workspace& ws, hipStream_t stream);

}  // namespace lrc

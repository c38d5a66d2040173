// Factor apply Y = U diag(s) (V^T X) and the FP64 product kernels of the
// matrix certificate, for gfx950.
//
// Apply (Sec. 4.4 eq. gpu_matrix_apply), two phases:
//   phase 1  T'^T[c][j] = s_j * sum_i V[i][j] X[i][c]   (sum split over i in a
//            fixed number of chunks, combined in chunk order by the last
//            workgroup to finish: deterministic, no floating-point atomics)
//   phase 2  Y[i][c]    = sum_j U[i][j] T'^T[c][j]
// T'^T is kept in the storage type: FP64 / FP32 accumulate and store in
// their own precision; FP16 accumulates in FP32 and rounds T' once to FP16
// because it is the FP16 input of the second matrix-core product.
//
// Two kernel pairs (regime dispatch):
//   streaming  batch <= 8: one lane per column of V (phase 1) and wavefront
//              dot products with a butterfly reduction over rows of U
//              (phase 2); the factors are read once, coalesced.
//   MFMA       otherwise: 64 x 64 output tiles on the 16x16 matrix cores
//              (f64 16x16x4, f32 16x16x4, f16 16x16x32 with FP32 accumulation),
//              operands staged through LDS, register double-buffered.
#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

// ------------------------------------------------------------ tile config --
template <typename T, int BM_, int BN_, int BK_, int WM_, int WN_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
    static constexpr int NT = WM * WN * 64;
    static constexpr int KPL = PrecTraits<T>::KPL, KB = PrecTraits<T>::KB;
    static constexpr int PAD = (KPL == 8) ? 8 : 1;   // keeps f16 rows 16-byte aligned
    static constexpr int LDK = BK + PAD;
    static constexpr int WTM = BM / WM, WTN = BN / WN;
    static constexpr int FM = WTM / 16, FN = WTN / 16;
    static constexpr int EA = BM * BK / NT, EB = BN * BK / NT;   // staged elements per thread
    using Acc = typename PrecTraits<T>::acc;
    using AccV = typename PrecTraits<T>::accv;
    using Frag = typename PrecTraits<T>::frag;
    static_assert(BK % KB == 0, "BK must be a multiple of the MFMA K step");
    static_assert(WTM % 16 == 0 && WTN % 16 == 0, "wave tile must be a multiple of 16");
    static_assert((BM * BK) % NT == 0 && (BN * BK) % NT == 0, "tile must split evenly");
};

template <typename T> struct ApplyCfg;
template <> struct ApplyCfg<double> { using C = Cfg<double, 64, 64, 16, 2, 2>; };
template <> struct ApplyCfg<float> { using C = Cfg<float, 64, 64, 16, 2, 2>; };
template <> struct ApplyCfg<half_t> { using C = Cfg<half_t, 64, 64, 32, 2, 2>; };

// One BK step of MFMAs on LDS tiles As[BM][LDK] (rows = m) and Bs[BN][LDK]
// (rows = n).  acc[fn][fm][v] = C[m = wm*WTM + fm*16 + (lane&15)]
//                                [n = wn*WTN + fn*16 + acc_row<T>(lane>>4, v)].
template <class C, typename T>
__device__ __forceinline__ void mma_tile(const T* As, const T* Bs, typename C::AccV (&acc)[C::FN][C::FM],
                                         int wm, int wn, int lane) {
    const int r = lane & 15, g = lane >> 4;
#pragma unroll
    for (int kk = 0; kk < C::BK; kk += C::KB) {
        typename C::Frag a[C::FN], b[C::FM];
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
            a[fn] = load_frag<T>(Bs + (wn * C::WTN + fn * 16 + r) * C::LDK + kk + g * C::KPL);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
            b[fm] = load_frag<T>(As + (wm * C::WTM + fm * 16 + r) * C::LDK + kk + g * C::KPL);
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = mfma(a[fn], b[fm], acc[fn][fm]);
    }
}

// Global -> registers for a ROWS x BK tile whose source is [K][ld] with the
// row index contiguous (a transposed read): consecutive threads read
// consecutive rows, i.e. consecutive addresses.
template <class C, int ROWS, int E, typename T>
__device__ __forceinline__ void fetch_rowm(T (&reg)[E], const T* __restrict__ src, int64_t ld,
                                           int64_t r0, int64_t rlim, int64_t k0, int64_t klim, int tid) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int idx = tid + e * C::NT;
        const int rr = idx % ROWS, kk = idx / ROWS;
        const int64_t gr = r0 + rr, gk = k0 + kk;
        reg[e] = (gr < rlim && gk < klim) ? src[gk * ld + gr] : T(0);
    }
}
template <class C, int ROWS, int E, typename T>
__device__ __forceinline__ void stash_rowm(T* S, const T (&reg)[E], int tid) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int idx = tid + e * C::NT;
        S[(idx % ROWS) * C::LDK + idx / ROWS] = reg[e];
    }
}
// Same for a source [rows][ld] with the K index contiguous.
template <class C, int ROWS, int E, typename T>
__device__ __forceinline__ void fetch_rowk(T (&reg)[E], const T* __restrict__ src, int64_t ld,
                                           int64_t r0, int64_t rlim, int64_t k0, int64_t klim, int tid) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int idx = tid + e * C::NT;
        const int kk = idx % C::BK, rr = idx / C::BK;
        const int64_t gr = r0 + rr, gk = k0 + kk;
        reg[e] = (gr < rlim && gk < klim) ? src[gr * ld + gk] : T(0);
    }
}
template <class C, int ROWS, int E, typename T>
__device__ __forceinline__ void stash_rowk(T* S, const T (&reg)[E], int tid) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int idx = tid + e * C::NT;
        S[(idx / C::BK) * C::LDK + idx % C::BK] = reg[e];
    }
}

enum { ATB_APPLY = 0, ATB_GRAM = 1 };

// C[m][n] = sum_{i in chunk} A[i][m] B[i][n]  (both sources [K][ld], row
// index contiguous).  Grid (tiles_n, tiles_m, splits).
//   ATB_APPLY: out is T'^T[n][ldo] in T, value s[m] * C (s[m] = 0 for m >= M),
//              written for m < Mout (zero padding rows included).
//   ATB_GRAM : out is G[m][ldo] in double (T = double).
template <typename T, class C, int MODE>
__global__ __launch_bounds__(C::NT) void k_atb(
    const T* __restrict__ Asrc, int64_t lda, const T* __restrict__ Bsrc, int64_t ldb,
    int64_t M, int64_t N, int64_t K, int64_t chunk, int splits,
    typename C::Acc* __restrict__ part, int* __restrict__ counters,
    const T* __restrict__ svals, void* __restrict__ out, int64_t ldo, int64_t Mout) {
    using Acc = typename C::Acc;
    using AccV = typename C::AccV;
    __shared__ alignas(16) T As[C::BM * C::LDK];
    __shared__ alignas(16) T Bs[C::BN * C::LDK];
    __shared__ int last_flag;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / C::WN, wn = wave % C::WN;
    const int64_t m0 = (int64_t)blockIdx.y * C::BM, n0 = (int64_t)blockIdx.x * C::BN;
    const int sp = blockIdx.z;
    const int64_t kbeg = (int64_t)sp * chunk;
    const int64_t kend = (kbeg + chunk < K) ? kbeg + chunk : K;

    AccV acc[C::FN][C::FM];
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = zero_accv<AccV>();

    T ra[C::EA], rb[C::EB];
    if (kbeg < kend) {
        fetch_rowm<C, C::BM>(ra, Asrc, lda, m0, M, kbeg, kend, tid);
        fetch_rowm<C, C::BN>(rb, Bsrc, ldb, n0, N, kbeg, kend, tid);
    }
    for (int64_t k0 = kbeg; k0 < kend; k0 += C::BK) {
        stash_rowm<C, C::BM>(As, ra, tid);
        stash_rowm<C, C::BN>(Bs, rb, tid);
        __syncthreads();
        if (k0 + C::BK < kend) {
            fetch_rowm<C, C::BM>(ra, Asrc, lda, m0, M, k0 + C::BK, kend, tid);
            fetch_rowm<C, C::BN>(rb, Bsrc, ldb, n0, N, k0 + C::BK, kend, tid);
        }
        mma_tile<C>(As, Bs, acc, wm, wn, lane);
        __syncthreads();
    }

    const int r = lane & 15, g = lane >> 4;
    if (splits > 1) {
        const int64_t tile = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
        constexpr int NV = C::FN * C::FM * 4;
        Acc* mine = part + ((tile * splits + sp) * NV) * C::NT;
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
                for (int v = 0; v < 4; ++v) mine[((fn * C::FM + fm) * 4 + v) * C::NT + tid] = acc[fn][fm][v];
        if (!arrive_last(counters + tile, splits, &last_flag)) return;
        // every partial, this workgroup's included, is read back in split order
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = zero_accv<AccV>();
        for (int q = 0; q < splits; ++q) {
            const Acc* src = part + ((tile * splits + q) * NV) * C::NT;
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
                for (int fm = 0; fm < C::FM; ++fm)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        acc[fn][fm][v] += __builtin_nontemporal_load(&src[((fn * C::FM + fm) * 4 + v) * C::NT + tid]);
        }
    }

#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) {
            const int64_t mm = m0 + wm * C::WTM + fm * 16 + r;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t nn = n0 + wn * C::WTN + fn * 16 + acc_row<T>(g, v);
                if (MODE == ATB_APPLY) {
                    if (nn < N && mm < Mout) {
                        const Acc sm = (mm < M) ? to_acc(svals[mm]) : Acc(0);
                        static_cast<T*>(out)[nn * ldo + mm] = to_storage<T>(sm * acc[fn][fm][v]);
                    }
                } else {
                    if (nn < N && mm < M) static_cast<double*>(out)[mm * ldo + nn] = (double)acc[fn][fm][v];
                }
            }
        }
}

enum { ABT_STORE = 0, ABT_ERR = 1 };

// C[m][n] = sum_k A[m][k] B[n][k]  (both sources with K contiguous).
// Grid (tiles_n, tiles_m).
//   ABT_STORE: Y[m][ldy] = C rounded to T.
//   ABT_ERR  : (T = double) partial sum of (Aref[m][n] - C)^2 per workgroup.
template <typename T, class C, int MODE>
__global__ __launch_bounds__(C::NT) void k_abt(
    const T* __restrict__ Asrc, int64_t lda, int64_t M, int64_t Ka,
    const T* __restrict__ Bsrc, int64_t ldb, int64_t N, int64_t Kb, int64_t K,
    T* __restrict__ Y, int64_t ldy, int vec4,
    const double* __restrict__ Aref, int64_t ldr, double* __restrict__ part) {
    using AccV = typename C::AccV;
    __shared__ alignas(16) T As[C::BM * C::LDK];
    __shared__ alignas(16) T Bs[C::BN * C::LDK];
    __shared__ double wsum[C::NT / 64];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / C::WN, wn = wave % C::WN;
    const int64_t m0 = (int64_t)blockIdx.y * C::BM, n0 = (int64_t)blockIdx.x * C::BN;

    AccV acc[C::FN][C::FM];
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = zero_accv<AccV>();

    T ra[C::EA], rb[C::EB];
    fetch_rowk<C, C::BM>(ra, Asrc, lda, m0, M, 0, Ka, tid);
    fetch_rowk<C, C::BN>(rb, Bsrc, ldb, n0, N, 0, Kb, tid);
    for (int64_t k0 = 0; k0 < K; k0 += C::BK) {
        stash_rowk<C, C::BM>(As, ra, tid);
        stash_rowk<C, C::BN>(Bs, rb, tid);
        __syncthreads();
        if (k0 + C::BK < K) {
            fetch_rowk<C, C::BM>(ra, Asrc, lda, m0, M, k0 + C::BK, Ka, tid);
            fetch_rowk<C, C::BN>(rb, Bsrc, ldb, n0, N, k0 + C::BK, Kb, tid);
        }
        mma_tile<C>(As, Bs, acc, wm, wn, lane);
        __syncthreads();
    }

    const int r = lane & 15, g = lane >> 4;
    if (MODE == ABT_STORE) {
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) {
                const int64_t mm = m0 + wm * C::WTM + fm * 16 + r;
                const int64_t nb = n0 + wn * C::WTN + fn * 16;
                if (mm >= M) continue;
                T* dst = Y + mm * ldy + nb;
                if (AccRowsContiguous<T>::value && vec4 && nb + 4 * g + 3 < N) {
                    typedef T vec_t __attribute__((ext_vector_type(4)));
                    vec_t w;
#pragma unroll
                    for (int v = 0; v < 4; ++v) w[v] = to_storage<T>(acc[fn][fm][v]);
                    *reinterpret_cast<vec_t*>(dst + 4 * g) = w;
                } else {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int row = acc_row<T>(g, v);
                        if (nb + row < N) dst[row] = to_storage<T>(acc[fn][fm][v]);
                    }
                }
            }
    } else {
        double sum = 0.0;
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) {
                const int64_t mm = m0 + wm * C::WTM + fm * 16 + r;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t nn = n0 + wn * C::WTN + fn * 16 + acc_row<T>(g, v);
                    if (mm < M && nn < N) {
                        const double dlt = Aref[mm * ldr + nn] - (double)acc[fn][fm][v];
                        sum += dlt * dlt;
                    }
                }
            }
        sum = wave_sum(sum);
        if (lane == 0) wsum[wave] = sum;
        __syncthreads();
        if (tid == 0) {
            double t = 0.0;
            for (int w = 0; w < C::NT / 64; ++w) t += wsum[w];
            part[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = t;
        }
    }
}

// --------------------------------------------------------- streaming path --
// Phase 1, batch <= NB: workgroup (jg, sp) owns columns [64 jg, 64 jg + 64)
// of V and rows [sp*chunk, (sp+1)*chunk) of V and X.  Lane j of every wave
// accumulates column j; the four waves take interleaved rows and are summed
// in wave order.  The last workgroup of each column group combines the
// per-chunk partials in chunk order, scales by s and writes T'^T.
template <typename T, int NB>
__global__ __launch_bounds__(256) void k_p1_stream(
    const T* __restrict__ V, const T* __restrict__ X, const T* __restrict__ s, T* __restrict__ Tt,
    int64_t ldt, typename PrecTraits<T>::acc* __restrict__ part, int* __restrict__ counters,
    int64_t n, int64_t k, int64_t b, int64_t chunk, int splits) {
    using Acc = typename PrecTraits<T>::acc;
    __shared__ Acc red[4][64][NB];
    __shared__ int last_flag;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int jg = blockIdx.x, sp = blockIdx.y;
    const int64_t j = (int64_t)jg * 64 + lane;
    const int64_t i0 = (int64_t)sp * chunk;
    const int64_t i1 = (i0 + chunk < n) ? i0 + chunk : n;

    Acc acc[NB];
#pragma unroll
    for (int c = 0; c < NB; ++c) acc[c] = 0;
    if (j < k) {
        for (int64_t i = i0 + wave; i < i1; i += 4) {
            const Acc vij = to_acc(V[i * k + j]);
#pragma unroll
            for (int c = 0; c < NB; ++c)
                if (c < b) acc[c] += vij * to_acc(X[i * b + c]);
        }
    }
#pragma unroll
    for (int c = 0; c < NB; ++c) red[wave][lane][c] = acc[c];
    __syncthreads();
    if (wave == 0) {
#pragma unroll
        for (int c = 0; c < NB; ++c) {
            const Acc t = ((red[0][lane][c] + red[1][lane][c]) + red[2][lane][c]) + red[3][lane][c];
            part[(((int64_t)jg * splits + sp) * 64 + lane) * NB + c] = t;
        }
    }
    if (!arrive_last(counters + jg, splits, &last_flag)) return;
    // columns of this group, including the zero rows j in [k, ldt) of T'^T
    for (int idx = tid; idx < 64 * NB; idx += 256) {
        const int jl = idx / NB, c = idx % NB;
        const int64_t jj = (int64_t)jg * 64 + jl;
        if (c >= b || jj >= ldt) continue;
        Acc sum = 0;
        if (jj < k) {
            for (int q = 0; q < splits; ++q)
                sum += __builtin_nontemporal_load(&part[(((int64_t)jg * splits + q) * 64 + jl) * NB + c]);
        }
        const Acc sj = (jj < k) ? to_acc(s[jj]) : Acc(0);
        Tt[(int64_t)c * ldt + jj] = to_storage<T>(sj * sum);
    }
}

// Phase 2, batch <= NB: T' staged in LDS (accumulation type); every wave
// takes 4 rows of U at a time, lanes stride over j, and a butterfly sum
// over the wave gives each output.
template <typename T, int NB>
__global__ __launch_bounds__(256) void k_p2_stream(
    const T* __restrict__ U, const T* __restrict__ Tt, int64_t ldt, T* __restrict__ Y,
    int64_t m, int64_t k, int64_t b) {
    using Acc = typename PrecTraits<T>::acc;
    extern __shared__ double4_t smem_v[];
    Acc* Ts = reinterpret_cast<Acc*>(smem_v);   // [k][NB]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int64_t idx = tid; idx < k * NB; idx += 256) {
        const int64_t jj = idx / NB;
        const int c = (int)(idx % NB);
        Ts[idx] = (c < b) ? to_acc(Tt[(int64_t)c * ldt + jj]) : Acc(0);
    }
    __syncthreads();
    constexpr int RPW = 4;
    const int64_t row0 = ((int64_t)blockIdx.x * 4 + wave) * RPW;
    Acc acc[RPW][NB];
#pragma unroll
    for (int q = 0; q < RPW; ++q)
#pragma unroll
        for (int c = 0; c < NB; ++c) acc[q][c] = 0;
    for (int64_t jj = lane; jj < k; jj += 64) {
#pragma unroll
        for (int q = 0; q < RPW; ++q) {
            const int64_t row = row0 + q;
            if (row < m) {
                const Acc u = to_acc(U[row * k + jj]);
#pragma unroll
                for (int c = 0; c < NB; ++c) acc[q][c] += u * Ts[jj * NB + c];
            }
        }
    }
#pragma unroll
    for (int q = 0; q < RPW; ++q)
#pragma unroll
        for (int c = 0; c < NB; ++c) acc[q][c] = wave_sum(acc[q][c]);
    if (lane == 0) {
#pragma unroll
        for (int q = 0; q < RPW; ++q) {
            const int64_t row = row0 + q;
            if (row < m)
                for (int c = 0; c < NB && c < b; ++c) Y[row * b + c] = to_storage<T>(acc[q][c]);
        }
    }
}

// ------------------------------------------------------------------- host --
static constexpr int kStreamMaxBatch = 8;
static constexpr int kStreamRowsTarget = 64;     // rows of V per workgroup chunk (phase 1)

ApplyPlan plan_apply(int64_t m, int64_t n, int64_t k, int64_t b, int prec, int path) {
    (void)m;
    ApplyPlan p{};
    if (path != 1 && path != 2) path = (b <= kStreamMaxBatch) ? 1 : 2;
    if (path == 1 && b > kStreamMaxBatch) path = 2;
    p.path = path;
    p.Kp = round_up(k, 8);
    const size_t acc_b = (prec == P64) ? 8 : 4;
    if (path == 1) {
        p.tiles_m = (int)((k + 63) / 64);
        p.tiles_n = 1;
        int64_t splits = (n + kStreamRowsTarget - 1) / kStreamRowsTarget;
        if (splits > 256) splits = 256;
        if (splits < 1) splits = 1;
        p.chunk = (n + splits - 1) / splits;
        p.splits = (int)((n + p.chunk - 1) / p.chunk);
        const int nb = (b <= 1) ? 1 : (b <= 2) ? 2 : (b <= 4) ? 4 : 8;
        p.part_bytes = (size_t)p.tiles_m * p.splits * 64 * nb * acc_b;
        p.counters = (size_t)p.tiles_m;
    } else {
        const int BK = (prec == P16) ? 32 : 16;
        p.tiles_m = (int)((k + 63) / 64);
        p.tiles_n = (int)((b + 63) / 64);
        const int64_t base = (int64_t)p.tiles_m * p.tiles_n;
        int64_t splits = (1024 + base - 1) / base;
        int64_t max_splits = n / (4 * BK);
        if (max_splits < 1) max_splits = 1;
        if (splits > max_splits) splits = max_splits;
        if (splits < 1) splits = 1;
        p.chunk = round_up((n + splits - 1) / splits, BK);
        p.splits = (int)((n + p.chunk - 1) / p.chunk);
        p.part_bytes = (p.splits > 1) ? (size_t)base * p.splits * 64 * 64 * acc_b : 0;
        p.counters = (p.splits > 1) ? (size_t)base : 0;
    }
    p.mid_bytes = (size_t)b * p.Kp * elem_bytes(prec);
    return p;
}

size_t apply_workspace_bytes(const ApplyPlan& p) {
    return round_up(p.part_bytes, 256) + round_up(p.mid_bytes, 256);
}

template <typename T> static const char* p1_stream_label();
template <typename T> static const char* p2_stream_label();
template <typename T> static const char* p1_mfma_label();
template <typename T> static const char* p2_mfma_label();
#define LRC_LABELS(T, S)                                                          \
    template <> const char* p1_stream_label<T>() { return "apply_p1_stream_" S; } \
    template <> const char* p2_stream_label<T>() { return "apply_p2_stream_" S; } \
    template <> const char* p1_mfma_label<T>() { return "apply_p1_mfma_" S; }     \
    template <> const char* p2_mfma_label<T>() { return "apply_p2_mfma_" S; }
LRC_LABELS(double, "f64")
LRC_LABELS(float, "f32")
LRC_LABELS(half_t, "f16")
#undef LRC_LABELS

template <typename T>
static hipError_t apply_typed(const ApplyPlan& p, const T* U, const T* s, const T* V, const T* X,
                              T* Y, int64_t m, int64_t n, int64_t k, int64_t b, Workspace& ws,
                              hipStream_t stream) {
    using Acc = typename PrecTraits<T>::acc;
    Acc* part = static_cast<Acc*>(ws.take(p.part_bytes));
    T* Tt = static_cast<T*>(ws.take(p.mid_bytes));
    int* counters = ws.counters;
    if (ws.overrun || !Tt || (p.counters && ws.n_counters < p.counters)) return hipErrorOutOfMemory;
    const int64_t ldt = p.Kp;
    if (p.path == 1) {
        dim3 g1(p.tiles_m, p.splits);
        {
            KernelTimer t1(p1_stream_label<T>(), stream);
#define LRC_P1S(NB) hipLaunchKernelGGL((k_p1_stream<T, NB>), g1, dim3(256), 0, stream, V, X, s, Tt, ldt, part, counters, n, k, b, p.chunk, p.splits)
            if (b <= 1) LRC_P1S(1); else if (b <= 2) LRC_P1S(2); else if (b <= 4) LRC_P1S(4); else LRC_P1S(8);
#undef LRC_P1S
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t rows_per_wg = 16;
        dim3 g2((unsigned)((m + rows_per_wg - 1) / rows_per_wg));
        KernelTimer t2(p2_stream_label<T>(), stream);
#define LRC_P2S(NB) hipLaunchKernelGGL((k_p2_stream<T, NB>), g2, dim3(256), (size_t)k * NB * sizeof(Acc), stream, U, Tt, ldt, Y, m, k, b)
        if (b <= 1) LRC_P2S(1); else if (b <= 2) LRC_P2S(2); else if (b <= 4) LRC_P2S(4); else LRC_P2S(8);
#undef LRC_P2S
        return hipGetLastError();
    }
    using C = typename ApplyCfg<T>::C;
    dim3 g1(p.tiles_n, p.tiles_m, p.splits);
    {
    KernelTimer t1(p1_mfma_label<T>(), stream);
    hipLaunchKernelGGL((k_atb<T, C, ATB_APPLY>), g1, dim3(C::NT), 0, stream, V, k, X, b, k, b, n,
                       p.chunk, p.splits, part, counters, s, (void*)Tt, ldt, ldt);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2((unsigned)((b + C::BN - 1) / C::BN), (unsigned)((m + C::BM - 1) / C::BM));
    KernelTimer t2(p2_mfma_label<T>(), stream);
    const int vec4 = (b % 4 == 0) && ((reinterpret_cast<uintptr_t>(Y) % (4 * sizeof(T))) == 0);
    hipLaunchKernelGGL((k_abt<T, C, ABT_STORE>), g2, dim3(C::NT), 0, stream, U, k, m, k, (const T*)Tt,
                       ldt, b, ldt, ldt, Y, b, vec4, (const double*)nullptr, (int64_t)0, (double*)nullptr);
    return hipGetLastError();
}

hipError_t launch_apply(const ApplyPlan& p, const void* U, const void* s, const void* V, const void* X,
                        void* Y, int64_t m, int64_t n, int64_t k, int64_t b, int prec, Workspace& ws,
                        hipStream_t stream) {
    switch (prec) {
    case P64:
        return apply_typed<double>(p, (const double*)U, (const double*)s, (const double*)V, (const double*)X,
                                   (double*)Y, m, n, k, b, ws, stream);
    case P32:
        return apply_typed<float>(p, (const float*)U, (const float*)s, (const float*)V, (const float*)X,
                                  (float*)Y, m, n, k, b, ws, stream);
    default:
        return apply_typed<half_t>(p, (const half_t*)U, (const half_t*)s, (const half_t*)V, (const half_t*)X,
                                   (half_t*)Y, m, n, k, b, ws, stream);
    }
}

// ----------------------------------------------------- certificate (FP64) --
using GramC = Cfg<double, 64, 64, 16, 2, 2>;

static void gram_plan(int64_t rows, int64_t cols, int* tiles, int* splits, int64_t* chunk) {
    const int t = (int)((cols + 63) / 64);
    const int64_t base = (int64_t)t * t;
    int64_t sp = (1024 + base - 1) / base;
    int64_t mx = rows / 64;
    if (mx < 1) mx = 1;
    if (sp > mx) sp = mx;
    if (sp < 1) sp = 1;
    *chunk = round_up((rows + sp - 1) / sp, 16);
    *splits = (int)((rows + *chunk - 1) / *chunk);
    *tiles = t;
}

size_t gram_workspace_bytes(int64_t rows, int64_t cols, size_t* counters) {
    int t, sp;
    int64_t ch;
    gram_plan(rows, cols, &t, &sp, &ch);
    *counters = (size_t)t * t;
    return (size_t)t * t * sp * 64 * 64 * sizeof(double);
}

hipError_t launch_gram(const double* P, int64_t rows, int64_t cols, double* G, Workspace& ws,
                       hipStream_t stream) {
    int t, sp;
    int64_t ch;
    gram_plan(rows, cols, &t, &sp, &ch);
    double* part = static_cast<double*>(ws.take((size_t)t * t * sp * 64 * 64 * sizeof(double)));
    if (ws.overrun || (sp > 1 && ws.n_counters < (size_t)t * t)) return hipErrorOutOfMemory;
    dim3 g(t, t, sp);
    KernelTimer tm("cert_gram_f64", stream);
    hipLaunchKernelGGL((k_atb<double, GramC, ATB_GRAM>), g, dim3(GramC::NT), 0, stream, P, cols, P, cols,
                       cols, cols, rows, ch, sp, part, ws.counters, (const double*)nullptr, (void*)G, cols,
                       cols);
    return hipGetLastError();
}

size_t err_workspace_bytes(int64_t m, int64_t n) {
    return (size_t)((m + 63) / 64) * ((n + 63) / 64) * sizeof(double);
}

hipError_t launch_err_dense(const double* A, const double* W, const double* Vw, int64_t m, int64_t n,
                            int64_t r, double* part, int64_t* nparts, hipStream_t stream) {
    dim3 g((unsigned)((n + 63) / 64), (unsigned)((m + 63) / 64));
    *nparts = (int64_t)g.x * g.y;
    const int64_t K = round_up(r, GramC::BK);
    KernelTimer tm("cert_err_dense_f64", stream);
    hipLaunchKernelGGL((k_abt<double, GramC, ABT_ERR>), g, dim3(GramC::NT), 0, stream, W, r, m, r, Vw, r, n, r,
                       K, (double*)nullptr, (int64_t)0, 0, A, n, part);
    return hipGetLastError();
}

}  // namespace lrc

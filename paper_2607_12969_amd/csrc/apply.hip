// Factor apply Y = U diag(s) (V^T X) and the FP64 product kernels of the
// matrix certificate, for gfx950.
//
// Apply (Sec. 4.4 eq. gpu_matrix_apply), two phases:
//   phase 1  T'^T[c][j] = s_j * sum_i V[i][j] X[i][c]   (sum split over i in a
//            fixed number of chunks whose partials a second kernel adds in
//            chunk order: deterministic, no floating-point atomics)
//   phase 2  Y[i][c]    = sum_j U[i][j] T'^T[c][j]
// T'^T is kept in the storage type: FP64 / FP32 accumulate and store in
// their own precision; FP16 accumulates in FP32 and rounds T' once to FP16
// because it is the FP16 input of the second matrix-core product.
//
// Two kernel pairs (regime dispatch):
//   streaming  batch <= 8: one lane per column of V (phase 1) and wavefront
//              dot products with a butterfly reduction over rows of U
//              (phase 2); the factors are read once, coalesced.
//   MFMA       otherwise: 128 x 128 (large shapes) or 64 x 64 output tiles
//              on the 16x16 matrix cores (f64 16x16x4, f32 16x16x4, f16
//              16x16x32 with FP32 accumulation); operands move in 16-byte
//              chunks (operands with an unaligned pitch are first copied
//              into a padded workspace), are staged through LDS with three
//              K steps of loads in flight; workgroups are renumbered so
//              that tiles sharing an operand run on the same XCD.
#include <cstdlib>
#include <type_traits>

#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

// ------------------------------------------------------------ tile config --
template <typename T, int BM_, int BN_, int BK_, int WM_, int WN_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_;
    static constexpr int NT = WM * WN * 64;
    static constexpr int KPL = PrecTraits<T>::KPL, KB = PrecTraits<T>::KB;
    static constexpr int VEC = 16 / (int)sizeof(T);       // elements per 16-byte access
    // tiles with K contiguous: [rows][BK + PADK]; rows stay 16-byte aligned
    // (fragments are read 16 bytes at a time) and start an odd number of
    // 16-byte chunks apart
    static constexpr int PADK = 16 / (int)sizeof(T);
    static constexpr int LDK = BK + PADK;
    // tiles with rows contiguous: [BK][rows + PADR]; the pad shifts successive
    // K rows across the LDS banks read by one fragment load
    static constexpr int PADR = (sizeof(T) == 8) ? 2 : 16;
    static constexpr int LDA_R = BM + PADR, LDB_R = BN + PADR;
    static constexpr int WTM = BM / WM, WTN = BN / WN;
    static constexpr int FM = WTM / 16, FN = WTN / 16;
    using Acc = typename PrecTraits<T>::acc;
    using AccV = typename PrecTraits<T>::accv;
    using Frag = typename PrecTraits<T>::frag;
    static_assert(BK % KB == 0, "BK must be a multiple of the MFMA K step");
    static_assert(WTM % 16 == 0 && WTN % 16 == 0, "wave tile must be a multiple of 16");
    static_assert((BM * BK) % (NT * VEC) == 0 && (BN * BK) % (NT * VEC) == 0, "tile must split evenly");
};

// large tiles for large problems, small tiles when a dimension is small
template <typename T> struct BigCfg;
// FP64 takes K steps of 8 with 128 x 128 tiles: its 128 accumulator
// registers per wave then fit beside the operands (240 VGPRs, two waves per
// SIMD for phase 2; K steps of 16 spill).  65536 x 4096, k = 512: phase 2
// 4.87 -> 4.78 ms, phase 1 344 -> 310 us; 8192^2, k = 256: 784 -> 735 us.
template <> struct BigCfg<double> { using C = Cfg<double, 128, 128, 8, 2, 2>; };
template <> struct BigCfg<float> { using C = Cfg<float, 128, 128, 16, 2, 2>; };
template <> struct BigCfg<half_t> { using C = Cfg<half_t, 128, 128, 32, 2, 2>; };
template <typename T> struct SmallCfg;
template <> struct SmallCfg<double> { using C = Cfg<double, 64, 64, 16, 2, 2>; };
template <> struct SmallCfg<float> { using C = Cfg<float, 64, 64, 16, 2, 2>; };
template <> struct SmallCfg<half_t> { using C = Cfg<half_t, 64, 64, 32, 2, 2>; };

// ---- global -> registers -> LDS tile movers ---------------------------------
// fetch() only issues loads into registers; stash() writes LDS.  Rows past
// the matrix edge are read from a clamped, in-bounds address and left
// unmasked: they only feed output rows / columns that are discarded (or
// forced to zero) at the epilogue.  The K range is exact: only the last
// step of a K range can be partial, and there the missing K values are
// zeroed.

// Every thread moves whole 16-byte chunks.  When the source has a 16-byte
// aligned base and a pitch that is a multiple of the chunk (MIS = false), a
// chunk that starts inside a row stays inside that row's pitch and is read
// directly.  Otherwise (MIS = true: odd ranks such as the compensated k + 1,
// odd batches, offset views) a thread's chunk starts anywhere: it reads the
// two aligned 16-byte chunks that cover it and funnel-shifts them into place
// when it writes LDS, so the operand is read in place at any pitch.  The
// second aligned chunk is read only when it still holds an element of the
// matrix (else the first is read twice); an aligned chunk that holds a
// valid element lies inside one page of the allocation.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// The 16 bytes that start `sh` bytes into lo, continued into hi (sh in
// [0, 16), a multiple of the element size).  Whole dwords are picked by
// selects over named words (no array, so nothing is promoted to memory, and
// no 64-bit shifts); a 2-byte remainder (binary16) is taken with
// v_alignbyte.
template <typename T>
__device__ __forceinline__ u32x4_t funnel16(u32x4_t lo, u32x4_t hi, int sh) {
    const int dq = sh >> 2;
    const unsigned d0 = lo[0], d1 = lo[1], d2 = lo[2], d3 = lo[3], d4 = hi[0], d5 = hi[1], d6 = hi[2], d7 = hi[3];
    const bool q1 = dq == 1, q2 = dq == 2, q3 = dq == 3;
    const unsigned w0 = q3 ? d3 : q2 ? d2 : q1 ? d1 : d0;
    const unsigned w1 = q3 ? d4 : q2 ? d3 : q1 ? d2 : d1;
    const unsigned w2 = q3 ? d5 : q2 ? d4 : q1 ? d3 : d2;
    const unsigned w3 = q3 ? d6 : q2 ? d5 : q1 ? d4 : d3;
    u32x4_t out;
    if constexpr (sizeof(T) >= 4) {
        out[0] = w0;
        out[1] = w1;
        out[2] = w2;
        out[3] = w3;
    } else {
        const unsigned w4 = q3 ? d7 : q2 ? d6 : q1 ? d5 : d4;
        const unsigned sb = (unsigned)(sh & 3);   // 0 or 2
        out[0] = __builtin_amdgcn_alignbyte(w1, w0, sb);
        out[1] = __builtin_amdgcn_alignbyte(w2, w1, sb);
        out[2] = __builtin_amdgcn_alignbyte(w3, w2, sb);
        out[3] = __builtin_amdgcn_alignbyte(w4, w3, sb);
    }
    return out;
}

// Loads of a chunk of 16 bytes of T that starts at element address `el`
// (any alignment); `last` is the matrix's last element.
template <typename T>
struct MisChunk {
    static constexpr int CH = 16 / (int)sizeof(T);
    u32x4_t lo, hi;
    int sh;
    __device__ __forceinline__ void fetch(const T* el, const T* last) {
        const int off = (int)(reinterpret_cast<uintptr_t>(el) & 15) / (int)sizeof(T);   // elements past the chunk start
        const T* pa = el - off;
        const T* ph = (pa + CH <= last) ? pa + CH : pa;
        sh = off * (int)sizeof(T);
        lo = *reinterpret_cast<const u32x4_t*>(pa);
        hi = *reinterpret_cast<const u32x4_t*>(ph);
    }
    template <typename V>
    __device__ __forceinline__ V value() const {
        return __builtin_bit_cast(V, funnel16<T>(lo, hi, sh));
    }
};

// A tile of BK x ROWS elements taken from a source laid out [K][ld] with the
// ROWS index contiguous, into LDS [BK][ROWS + PADR].
template <class C, int ROWS, typename T, bool MIS = false>
struct RowsTile {
    static constexpr int CH = C::VEC;                            // elements per move
    static constexpr int E = C::BK * ROWS / (C::NT * CH);        // moves per thread
    static constexpr int LD = ROWS + C::PADR;                    // LDS pitch
    static constexpr int RC = ROWS / CH;                         // moves per K row
    static constexpr int KS = C::NT / RC;                        // K rows between a thread's moves
    static_assert(C::NT % RC == 0, "a thread keeps one column position");
    typedef T vec_t __attribute__((ext_vector_type(CH)));
    vec_t reg[MIS ? 1 : E];
    MisChunk<T> mc[MIS ? E : 1];
    // per-thread geometry: K row of move 0 and element offset of its column
    struct Geo {
        const T* base;   // source + r0 (uniform)
        int64_t ld;
        int kk0;         // K row of move 0 within a step
        int col;         // column offset within the tile, clamped into the matrix
        int lcol;        // LDS column of this thread
        const T* last;   // last element of the matrix (MIS)
    };
    __device__ __forceinline__ static Geo geo(const T* src, int64_t ld, int64_t r0, int64_t rlim, int tid,
                                              const T* last = nullptr) {
        Geo g;
        g.base = src + r0;
        g.ld = ld;
        g.kk0 = tid / RC;
        g.lcol = (tid % RC) * CH;
        g.col = (r0 + g.lcol < rlim) ? g.lcol : 0;
        g.last = last;
        return g;
    }
    __device__ __forceinline__ void fetch(const Geo& g, int64_t k0, bool partial, int64_t klim) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            int64_t gk = k0 + g.kk0 + e * KS;
            if (partial) gk = gk < klim ? gk : klim - 1;
            const T* p = g.base + gk * g.ld + g.col;
            if constexpr (MIS) mc[e].fetch(p, g.last);
            else reg[e] = *reinterpret_cast<const vec_t*>(p);
        }
    }
    __device__ __forceinline__ void stash(T* S, const Geo& g, int64_t k0, bool partial, int64_t klim) const {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int kk = g.kk0 + e * KS;
            vec_t w;
            if constexpr (MIS) w = mc[e].template value<vec_t>();
            else w = reg[e];
            if (partial && k0 + kk >= klim) {
#pragma unroll
                for (int v = 0; v < CH; ++v) w[v] = T(0);
            }
            *reinterpret_cast<vec_t*>(S + kk * LD + g.lcol) = w;
        }
    }
};

// A tile of ROWS x BK elements from a source laid out [rows][ld] with K
// contiguous, into LDS [ROWS][LDK].
template <class C, int ROWS, typename T, bool MIS = false>
struct KTile {
    static constexpr int CH = C::VEC;
    static constexpr int E = C::BK * ROWS / (C::NT * CH);
    static constexpr int KC = C::BK / CH;                        // moves per row
    static constexpr int RS = C::NT / KC;                        // rows between a thread's moves
    static_assert(C::NT % KC == 0, "a thread keeps one K position");
    typedef T vec_t __attribute__((ext_vector_type(CH)));
    vec_t reg[MIS ? 1 : E];
    MisChunk<T> mc[MIS ? E : 1];
    struct Geo {
        const T* base;   // source + r0 * ld (uniform)
        int64_t ld;
        int rr0;         // row of move 0 within the tile
        int rmax;        // last row inside the matrix, relative to r0
        int kq;          // K offset of this thread within a step
        const T* last;   // last element of the matrix (MIS)
    };
    __device__ __forceinline__ static Geo geo(const T* src, int64_t ld, int64_t r0, int64_t rlim, int tid,
                                              const T* last = nullptr) {
        Geo g;
        g.base = src + r0 * ld;
        g.ld = ld;
        g.rr0 = tid / KC;
        g.kq = (tid % KC) * CH;
        const int64_t rm = rlim - 1 - r0;
        g.rmax = rm < ROWS ? (int)rm : ROWS;
        g.last = last;
        return g;
    }
    __device__ __forceinline__ void fetch(const Geo& g, int64_t k0, bool partial, int64_t klim) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            int rr = g.rr0 + e * RS;
            rr = rr < g.rmax ? rr : g.rmax;
            int64_t gk = k0 + g.kq;
            if (partial && gk >= klim) gk = 0;
            const T* p = g.base + (int64_t)rr * g.ld + gk;
            if constexpr (MIS) mc[e].fetch(p, g.last);
            else reg[e] = *reinterpret_cast<const vec_t*>(p);
        }
    }
    __device__ __forceinline__ void stash(T* S, const Geo& g, int64_t k0, bool partial, int64_t klim) const {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const int rr = g.rr0 + e * RS;
            vec_t w;
            if constexpr (MIS) w = mc[e].template value<vec_t>();
            else w = reg[e];
            if (partial) {
                const int64_t gk = k0 + g.kq;
#pragma unroll
                for (int v = 0; v < CH; ++v)
                    if (gk + v >= klim) w[v] = T(0);
            }
            T* dst = S + rr * C::LDK + g.kq;
            if constexpr ((C::LDK * sizeof(T)) % 16 == 0) {
                *reinterpret_cast<vec_t*>(dst) = w;
            } else {
#pragma unroll
                for (int v = 0; v < CH; ++v) dst[v] = w[v];
            }
        }
    }
};

// MFMA operand fragment from a [BK][LD] (rows contiguous) tile for the 16
// rows starting at `rbase`; k0 is the first K value of this lane's slice.
// FP64 / FP32 take one K value per lane: a single LDS read.  FP16 takes 8
// consecutive K values of one row, which lie in 8 different LDS rows; two
// transposing LDS reads (ds_read_b64_tr_b16) gather them.  Within each group
// of 16 lanes, lane s points at the 4 consecutive rows 4(s&3).. of K row
// k0 + (s>>2); the instruction then returns to lane i the value of row i
// from the K rows addressed by lanes i/4, i/4+4, i/4+8, i/4+12, i.e. K
// values k0..k0+3 of its own row (a second read covers k0+4..k0+7).
template <typename T, int LD>
__device__ __forceinline__ typename PrecTraits<T>::frag frag_rows(const T* S, int rbase, int k0, int lane) {
    if constexpr (PrecTraits<T>::KPL == 1) {
        return S[k0 * LD + rbase + (lane & 15)];
    } else {
        static_assert(PrecTraits<T>::KPL == 8 && LD % 4 == 0, "transposing read needs 8-byte aligned rows");
        typedef short s4_t __attribute__((ext_vector_type(4)));
        const int s = lane & 15;
        const T* p = S + (k0 + (s >> 2)) * LD + rbase + 4 * (s & 3);
        const s4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4_t*)(p));
        const s4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4_t*)(p + 4 * LD));
        typedef short s8_t __attribute__((ext_vector_type(8)));
        const s8_t both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(typename PrecTraits<T>::frag, both);
    }
}

// One BK step of MFMAs.  Rows-contiguous tiles (phase 1, Gram):
// acc[fn][fm][v] = C[m = wm*WTM + fm*16 + (lane&15)][n = wn*WTN + fn*16 + acc_row<T>(lane>>4, v)]
// Fragments whose 16 rows (columns) all lie past the matrix edge are
// skipped: nfm / nfn count the live ones of this wave (wave-uniform).  Only
// edge tiles take the guarded form; interior tiles run branch-free.
template <class C, bool GUARD, typename T>
__device__ __forceinline__ void mma_rows_g(const T* As, const T* Bs, typename C::AccV (&acc)[C::FN][C::FM],
                                           int wm, int wn, int lane, int nfm, int nfn) {
    const int g = lane >> 4;
#pragma unroll
    for (int kk = 0; kk < C::BK; kk += C::KB) {
        typename C::Frag a[C::FN], b[C::FM];
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
            if (!GUARD || fn < nfn) a[fn] = frag_rows<T, C::LDB_R>(Bs, wn * C::WTN + fn * 16, kk + g * C::KPL, lane);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
            if (!GUARD || fm < nfm) b[fm] = frag_rows<T, C::LDA_R>(As, wm * C::WTM + fm * 16, kk + g * C::KPL, lane);
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                if (!GUARD || (fn < nfn && fm < nfm)) acc[fn][fm] = mfma(a[fn], b[fm], acc[fn][fm]);
    }
}

// Same for K-contiguous tiles As[BM][LDK], Bs[BN][LDK] (phase 2, error norm).
// FP64 and FP32 take one K value per lane and MFMA; a lane reads the RV =
// 16 / sizeof(T) consecutive values of its row at K offset RV g with one
// 16-byte LDS read and feeds value j to the j-th of RV MFMAs, so that MFMA j
// of a K block of 4 RV sums over k = RV g + j (the K values are taken in
// another order; every product is still added once).
template <class C, bool GUARD, typename T>
__device__ __forceinline__ void mma_k_g(const T* As, const T* Bs, typename C::AccV (&acc)[C::FN][C::FM], int wm,
                                        int wn, int lane, int nfm, int nfn) {
    const int r = lane & 15, g = lane >> 4;
    if constexpr (C::KPL == 1) {
        constexpr int RV = 16 / (int)sizeof(T);
        static_assert(C::BK % (C::KB * RV) == 0 && (C::LDK * sizeof(T)) % 16 == 0, "16-byte fragment reads");
        typedef T rv_t __attribute__((ext_vector_type(RV)));
#pragma unroll
        for (int kk = 0; kk < C::BK; kk += C::KB * RV) {
            rv_t a[C::FN], b[C::FM];
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn)
                if (!GUARD || fn < nfn)
                    a[fn] = *reinterpret_cast<const rv_t*>(Bs + (wn * C::WTN + fn * 16 + r) * C::LDK + kk + g * RV);
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                if (!GUARD || fm < nfm)
                    b[fm] = *reinterpret_cast<const rv_t*>(As + (wm * C::WTM + fm * 16 + r) * C::LDK + kk + g * RV);
#pragma unroll
            for (int j = 0; j < RV; ++j)
#pragma unroll
                for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
                    for (int fm = 0; fm < C::FM; ++fm)
                        if (!GUARD || (fn < nfn && fm < nfm)) acc[fn][fm] = mfma(a[fn][j], b[fm][j], acc[fn][fm]);
        }
        return;
    }
#pragma unroll
    for (int kk = 0; kk < C::BK; kk += C::KB) {
        typename C::Frag a[C::FN], b[C::FM];
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
            if (!GUARD || fn < nfn) a[fn] = load_frag<T>(Bs + (wn * C::WTN + fn * 16 + r) * C::LDK + kk + g * C::KPL);
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
            if (!GUARD || fm < nfm) b[fm] = load_frag<T>(As + (wm * C::WTM + fm * 16 + r) * C::LDK + kk + g * C::KPL);
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm)
                if (!GUARD || (fn < nfn && fm < nfm)) acc[fn][fm] = mfma(a[fn], b[fm], acc[fn][fm]);
    }
}


// Logical tiles of k_abt: groups of G = ceil(tiles_n / 8) n tiles, one group
// per XCD; inside a group n runs fastest, so consecutive workgroups share
// the rows of A, while the group's G column tiles of B stay in the L2.
struct AbtOrder {
    int64_t G, per_group, total;
    __host__ __device__ AbtOrder(int tiles_m, int tiles_n) {
        G = (tiles_n + 7) / 8;
        per_group = (int64_t)tiles_m * G;
        total = per_group * ((tiles_n + G - 1) / G);
    }
};

// live 16-wide fragments of a wave tile starting at `start` in a dimension of `lim`
template <int F>
__device__ __forceinline__ int live_frags(int64_t start, int64_t lim) {
    const int64_t rem = lim - start;
    if (rem <= 0) return 0;
    const int64_t f = (rem + 15) / 16;
    return f < F ? (int)f : F;
}

// Main loop shared by the tile kernels: K steps j = 0 .. nsteps-1 with two
// register stages of global loads and two LDS buffers.  Step s lives in
// register stage s % 2 and LDS buffer s % 2; iteration j multiplies buffer
// j % 2 while step j + 1 is written to the other buffer and the loads of
// step j + 3 are issued, so one barrier per step suffices and each load has
// two steps of matrix-core work to arrive.  Steps past the end are fetched
// from clamped addresses (never stashed), so every path issues the same
// loads and the compiler's waits cover exactly one stage.
// The pairs of steps run in a loop whose matrix-core work is unconditional
// (a conditional product inside it made the compiler keep two copies of the
// accumulators and move one into the other, behind a drain of the matrix
// pipeline, every step); an odd last step follows the loop.
template <bool PEEL, class Fetch, class Stash, class Mma>
__device__ __forceinline__ void pipeline2(int nsteps, int nfull, Fetch&& fetch, Stash&& stash, Mma&& mma) {
    if constexpr (!PEEL) nfull = 0;
    // fetch / stash take std::true_type for steps known to lie inside K
    // (nfull of them): no edge tests, so the loop body stays one block
    const std::false_type edge{};
    const std::true_type inside{};
    fetch(0, 0, edge);
    fetch(1, 1, edge);
    stash(0, 0, 0, edge);
    fetch(0, 2, edge);
    __syncthreads();
    int j = 0;
    for (; j + 4 < nfull; j += 2) {
        mma(0);
        stash(1, 1, j + 1, inside);
        fetch(1, j + 3, inside);
        __syncthreads();
        mma(1);
        stash(0, 0, j + 2, inside);
        fetch(0, j + 4, inside);
        __syncthreads();
    }
    for (; j + 1 < nsteps; j += 2) {
        // even step j: buffer 0; odd step j + 1: buffer 1
        mma(0);
        stash(1, 1, j + 1, edge);
        fetch(1, j + 3, edge);
        __syncthreads();
        mma(1);
        if (j + 2 < nsteps) stash(0, 0, j + 2, edge);
        fetch(0, j + 4, edge);
        __syncthreads();
    }
    if (j < nsteps) {
        mma(0);
        fetch(1, j + 3, edge);
        __syncthreads();
    }
}

// Whether the K-contiguous GEMM (phase 2) runs its inner steps edge-free:
// FP32 phase 2 2.57 -> 2.35 ms at 65536 x 4096; FP64 4.73 -> 4.33 ms, once
// the kernel is held to two waves per SIMD (the edge-free loop took 258
// registers, one wave per SIMD, and was 9 % slower than the single loop).
// The FP64 tile that reads a misaligned operand in place keeps the single
// loop and its own register budget: held to two waves it spills.
template <typename T, bool MIS = false>
constexpr bool kPeelAbt = sizeof(T) != 8 || !MIS;
template <typename T, bool MIS = false>
constexpr int kAbtMinWaves = kPeelAbt<T, MIS> ? 2 : 1;

// Calls f(std::false_type) for a tile whose fragments are all live (the
// branch-free products) and f(std::true_type) otherwise, so that the K loop
// itself carries no such branch.
template <class F>
__device__ __forceinline__ void by_edge(bool full, F&& f) {
    if (full) f(std::false_type{});
    else f(std::true_type{});
}

enum { ATB_APPLY = 0, ATB_GRAM = 1 };

// Store one finished fragment of C = A^T B (thread tid of the tile's
// workgroup, fragment (fn, fm), tile origin (m0, n0)).
//   ATB_APPLY: T'^T[n][ldo] = s[m] * C rounded to T, for m < Mout; rows
//              m >= M are written as zeros (their accumulators hold data of
//              clamped rows).
//   ATB_GRAM : G = P^T P is symmetric: only tiles on or above the diagonal
//              are computed, and the value of (m, n), m <= n, is written to
//              both G[m][n] and G[n][m] (T = double).
template <typename T, class C, int MODE>
__device__ __forceinline__ void atb_store(const typename C::AccV& a, int tid, int fn, int fm, int64_t m0,
                                          int64_t n0, int64_t M, int64_t N, const T* __restrict__ svals,
                                          void* __restrict__ out, int64_t ldo, int64_t Mout) {
    using Acc = typename C::Acc;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave / C::WN, wn = wave % C::WN;
    const int r = lane & 15, g = lane >> 4;
    const int64_t mm = m0 + wm * C::WTM + fm * 16 + r;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int64_t nn = n0 + wn * C::WTN + fn * 16 + acc_row<T>(g, v);
        if (MODE == ATB_APPLY) {
            if (nn < N && mm < Mout) {
                const Acc val = (mm < M) ? (svals ? to_acc(svals[mm]) * a[v] : a[v]) : Acc(0);
                static_cast<T*>(out)[nn * ldo + mm] = to_storage<T>(val);
            }
        } else {
            if (nn < N && mm < M && mm <= nn) {
                static_cast<double*>(out)[mm * ldo + nn] = (double)a[v];
                static_cast<double*>(out)[nn * ldo + mm] = (double)a[v];
            }
        }
    }
}

// C[m][n] = sum_{i in chunk} A[i][m] B[i][n]  (both sources [K][ld], row
// index contiguous).  One workgroup per (tile, split).  With one split the
// workgroup stores its tile (atb_store); otherwise it writes a partial tile
// and k_atb_finish, launched next on the same stream, sums them.  Kernel
// boundaries order the partials: no device-scope fences, which on this
// chip write back and invalidate the L2 of the XCD.
//   ATB_APPLY: out is T'^T[n][ldo] in T, value s[m] * C (s[m] = 0 for m >= M;
//              factor 1 when s is null),
//              written for m < Mout (zero padding rows included).
//   ATB_GRAM : out is G[m][ldo] in double (T = double).
// MIS: A has a misaligned base or pitch and is read in place; B is aligned.
template <typename T, class C, int MODE, bool MIS = false>
__global__ __launch_bounds__(C::NT) void k_atb(
    const T* __restrict__ Asrc, int64_t lda, const T* __restrict__ Bsrc, int64_t ldb,
    int64_t M, int64_t N, int64_t K, int64_t chunk, int tiles_m, int tiles_n, int splits,
    typename C::Acc* __restrict__ part, const T* __restrict__ svals, void* __restrict__ out, int64_t ldo,
    int64_t Mout) {
    using AccV = typename C::AccV;
    __shared__ alignas(16) T As[2][C::BK * C::LDA_R];
    __shared__ alignas(16) T Bs[2][C::BK * C::LDB_R];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / C::WN, wn = wave % C::WN;
    // logical order: m tile fastest (tiles sharing a block of B columns are neighbours), then n, then split
    const int64_t lt = xcd_tile((int64_t)tiles_m * tiles_n * splits);
    if (lt >= (int64_t)tiles_m * tiles_n * splits) return;
    const int64_t tile = lt % ((int64_t)tiles_m * tiles_n);
    const int sp = (int)(lt / ((int64_t)tiles_m * tiles_n));
    if (MODE == ATB_GRAM && tile % tiles_m > tile / tiles_m) return;   // below the diagonal
    const int64_t m0 = (tile % tiles_m) * C::BM, n0 = (tile / tiles_m) * C::BN;
    const int nfm = live_frags<C::FM>(m0 + wm * C::WTM, M), nfn = live_frags<C::FN>(n0 + wn * C::WTN, N);
    const int64_t kbeg = (int64_t)sp * chunk;
    const int64_t kend = (kbeg + chunk < K) ? kbeg + chunk : K;

    AccV acc[C::FN][C::FM];
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = zero_accv<AccV>();

    using TA = RowsTile<C, C::BM, T, MIS>;
    using TB = RowsTile<C, C::BN, T>;   // X (or the certificate's factor): aligned rows
    const typename TA::Geo ga = TA::geo(Asrc, lda, m0, M, tid, Asrc + (K - 1) * lda + (M - 1));
    const typename TB::Geo gb = TB::geo(Bsrc, ldb, n0, N, tid);
    TA ta[2];
    TB tb[2];
    const int nsteps = (int)((kend - kbeg + C::BK - 1) / C::BK);
    by_edge(nfm == C::FM && nfn == C::FN, [&](auto edge) {
        pipeline2<true>(
            nsteps, (int)((kend - kbeg) / C::BK),
            [&](int st, int j, auto in) {
                const int64_t k0 = kbeg + (int64_t)j * C::BK;
                const bool pk = !decltype(in)::value && k0 + C::BK > kend;
                ta[st].fetch(ga, k0, pk, kend);
                tb[st].fetch(gb, k0, pk, kend);
            },
            [&](int st, int buf, int j, auto in) {
                const int64_t k0 = kbeg + (int64_t)j * C::BK;
                const bool pk = !decltype(in)::value && k0 + C::BK > kend;
                ta[st].stash(As[buf], ga, k0, pk, kend);
                tb[st].stash(Bs[buf], gb, k0, pk, kend);
            },
            [&](int buf) { mma_rows_g<C, decltype(edge)::value>(As[buf], Bs[buf], acc, wm, wn, lane, nfm, nfn); });
    });

    if (splits > 1) {
        // partial tile: one accumulator vector per fragment, consecutive
        // threads on consecutive vectors; k_atb_finish sums the splits
        constexpr int NF = C::FN * C::FM;
        AccV* mine = reinterpret_cast<AccV*>(part) + ((tile * splits + sp) * NF) * C::NT + tid;
#pragma unroll
        for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
            for (int fm = 0; fm < C::FM; ++fm) mine[(fn * C::FM + fm) * C::NT] = acc[fn][fm];
        return;
    }
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm)
            atb_store<T, C, MODE>(acc[fn][fm], tid, fn, fm, m0, n0, M, N, svals, out, ldo, Mout);
}

// Sum of the split partials of k_atb, then the same store.  Workgroup
// (tile, fragment, slice) owns 64 consecutive thread positions of the tile's
// workgroups; its eight waves add eight consecutive runs of splits (each in
// split order, 16 loads in flight) and wave 0 adds the run sums in run
// order: a fixed order, with an eighth of the serial load chain.
constexpr int kFinishRuns = 8;

template <typename T, class C, int MODE>
__global__ __launch_bounds__(64 * kFinishRuns) void k_atb_finish(
    const typename C::AccV* __restrict__ part, int64_t M, int64_t N, int tiles_m, int splits,
    const T* __restrict__ svals, void* __restrict__ out, int64_t ldo, int64_t Mout) {
    using AccV = typename C::AccV;
    constexpr int NF = C::FN * C::FM, PQ = C::NT / 64;
    __shared__ AccV red[kFinishRuns][64];
    const int pl = threadIdx.x & 63;
    const int run = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t tile = blockIdx.x / (NF * PQ);
    const int f = (int)((blockIdx.x / PQ) % NF);
    const int pos = (int)(blockIdx.x % PQ) * 64 + pl;    // thread of the producing workgroup
    if (MODE == ATB_GRAM && tile % tiles_m > tile / tiles_m) return;   // below the diagonal
    const AccV* src = part + (tile * splits * NF + f) * C::NT + pos;
    const int64_t qs = (int64_t)NF * C::NT;      // stride between splits
    const int per = (splits + kFinishRuns - 1) / kFinishRuns;
    const int q0 = run * per < splits ? run * per : splits;
    const int q1 = q0 + per < splits ? q0 + per : splits;
    AccV acc = zero_accv<AccV>();
    int q = q0;
    for (; q + 16 <= q1; q += 16) {
        AccV pv[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) pv[u] = __builtin_nontemporal_load(src + (q + u) * qs);
#pragma unroll
        for (int u = 0; u < 16; ++u) acc += pv[u];
    }
    for (; q < q1; ++q) acc += __builtin_nontemporal_load(src + q * qs);
    red[run][pl] = acc;
    __syncthreads();
    if (run != 0) return;
    AccV sum = red[0][pl];
#pragma unroll
    for (int r = 1; r < kFinishRuns; ++r) sum += red[r][pl];
    const int64_t m0 = (tile % tiles_m) * C::BM, n0 = (tile / tiles_m) * C::BN;
    atb_store<T, C, MODE>(sum, pos, f / C::FM, f % C::FM, m0, n0, M, N, svals, out, ldo, Mout);
}

enum { ABT_STORE = 0, ABT_ERR = 1 };

// Output tile of k_abt rounded to T and written through LDS: the MFMA
// layout leaves each lane with 4 elements of one row, so direct stores
// would cover 16 rows x 32-64 bytes per instruction; staged, every lane
// writes 16 bytes and a wave writes whole row segments of the tile
// (BN * sizeof(T) bytes each), marked nontemporal since nothing here reads
// Y again.  The tile goes through in bands of rows
// (all BM rows at once when they fit the operand buffers that `stg` spans,
// else a wave row of WTM rows, or the largest half or quarter of one that
// fits, per band).  Rows >= M and columns >= N are not written.  vec16: Y
// and its pitch allow 16-byte stores.
template <typename T, class C>
__device__ __forceinline__ void abt_store_staged(const typename C::AccV (&acc)[C::FN][C::FM], T* stg, int tid,
                                                 int wm, int wn, int64_t m0, int64_t n0, int64_t M, int64_t N,
                                                 T* __restrict__ Y, int64_t ldy, int vec16) {
    constexpr int VEC = C::VEC;
    constexpr int LDS_ = C::BN + VEC;   // staged row pitch, 16-byte aligned
    constexpr int CAP = 2 * (C::BM + C::BN) * C::LDK;   // elements the operand buffers hold
    // rows per band: the whole tile, else the largest of a wave row, half
    // of one, a quarter of one, ... (down to one fragment) that fits
    constexpr int RB = C::BM * LDS_ <= CAP          ? C::BM
                       : C::WTM * LDS_ <= CAP       ? C::WTM
                       : (C::WTM / 2) * LDS_ <= CAP ? C::WTM / 2
                       : (C::WTM / 4) * LDS_ <= CAP ? C::WTM / 4
                                                    : 16;
    static_assert(RB >= 16 && RB * LDS_ <= CAP, "staging band exceeds the operand buffers");
    static_assert(RB == C::BM || C::WTM % RB == 0, "bands split wave rows evenly");
    static_assert(C::NT % (C::BN / VEC) == 0 && RB % (C::NT / (C::BN / VEC)) == 0, "band must split evenly");
    constexpr int CPR = C::BN / VEC;       // 16-byte chunks per row
    constexpr int RPP = C::NT / CPR;       // rows per pass
    const int lane = tid & 63, r = lane & 15, g = lane >> 4;
    typedef T vec_t __attribute__((ext_vector_type(VEC)));
#pragma unroll
    for (int band = 0; band < C::BM / RB; ++band) {
        if (band > 0) __syncthreads();   // the previous band has been read
        // tile rows [band RB, band RB + RB): staged by the waves of that wave
        // row, each writing its fragments that fall in the band
        const int lo = band * RB - wm * C::WTM;   // band start within this wave's rows
        if (RB == C::BM || (lo >= 0 && lo < C::WTM)) {
#pragma unroll
            for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
                for (int fm = 0; fm < C::FM; ++fm) {
                    const int srow = (RB == C::BM) ? wm * C::WTM + fm * 16 : fm * 16 - lo;
                    if (RB != C::BM && (srow < 0 || srow >= RB)) continue;
                    T* d = stg + (srow + r) * LDS_ + wn * C::WTN + fn * 16;
                    if (AccRowsContiguous<T>::value) {
                        typedef T v4_t __attribute__((ext_vector_type(4)));
                        v4_t w;
#pragma unroll
                        for (int v = 0; v < 4; ++v) w[v] = to_storage<T>(acc[fn][fm][v]);
                        *reinterpret_cast<v4_t*>(d + 4 * g) = w;
                    } else {
#pragma unroll
                        for (int v = 0; v < 4; ++v) d[acc_row<T>(g, v)] = to_storage<T>(acc[fn][fm][v]);
                    }
                }
        }
        __syncthreads();
        const int c = (tid % CPR) * VEC;
        const int64_t nn = n0 + c;
#pragma unroll
        for (int p = 0; p < RB / RPP; ++p) {
            const int row = p * RPP + tid / CPR;
            const int64_t mm = m0 + band * RB + row;
            if (mm >= M) break;
            const T* srow = stg + row * LDS_ + c;
            T* dst = Y + mm * ldy + nn;
            if (vec16 && nn + VEC <= N) {
                __builtin_nontemporal_store(*reinterpret_cast<const vec_t*>(srow), reinterpret_cast<vec_t*>(dst));
            } else {
#pragma unroll
                for (int v = 0; v < VEC; ++v)
                    if (nn + v < N) dst[v] = srow[v];
            }
        }
    }
}

// C[m][n] = sum_k A[m][k] B[n][k]  (both sources with K contiguous).
// One workgroup per tile, in the order of AbtOrder.
//   ABT_STORE: Y[m][ldy] = C rounded to T.
//   ABT_ERR  : (T = double) partial sum of (Aref[m][n] - C)^2 per workgroup.
template <typename T, class C, int MODE, bool MIS = false>
__global__ __launch_bounds__(C::NT, (kAbtMinWaves<T, MIS>)) void k_abt(
    const T* __restrict__ Asrc, int64_t lda, int64_t M, int64_t Ka,
    const T* __restrict__ Bsrc, int64_t ldb, int64_t N, int64_t Kb, int64_t K, int tiles_m, int tiles_n,
    T* __restrict__ Y, int64_t ldy, int vec16,
    const double* __restrict__ Aref, int64_t ldr, double* __restrict__ part) {
    using AccV = typename C::AccV;
    // both operand double buffers in one array: the store epilogue reuses it
    constexpr int kAs = C::BM * C::LDK, kBs = C::BN * C::LDK;
    __shared__ alignas(16) T smem[2 * kAs + 2 * kBs];
    __shared__ double wsum[C::NT / 64];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / C::WN, wn = wave % C::WN;
    const AbtOrder ord(tiles_m, tiles_n);
    const int64_t lt = xcd_tile(ord.total);
    if (lt >= ord.total) return;
    const int64_t mt = (lt % ord.per_group) / ord.G;
    const int64_t nt = (lt / ord.per_group) * ord.G + (lt % ord.per_group) % ord.G;
    if (nt >= tiles_n) return;
    const int64_t tile = mt * tiles_n + nt;
    const int64_t m0 = mt * C::BM, n0 = nt * C::BN;
    const int nfm = live_frags<C::FM>(m0 + wm * C::WTM, M), nfn = live_frags<C::FN>(n0 + wn * C::WTN, N);

    AccV acc[C::FN][C::FM];
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = zero_accv<AccV>();

    using TA = KTile<C, C::BM, T, MIS>;
    using TB = KTile<C, C::BN, T>;   // T'^T (or the certificate's factors): aligned rows
    const typename TA::Geo ga = TA::geo(Asrc, lda, m0, M, tid, Asrc + (M - 1) * lda + (Ka - 1));
    const typename TB::Geo gb = TB::geo(Bsrc, ldb, n0, N, tid);
    TA ta[2];
    TB tb[2];
    const int nsteps = (int)((K + C::BK - 1) / C::BK);
    by_edge(nfm == C::FM && nfn == C::FN, [&](auto edge) {
        pipeline2<kPeelAbt<T, MIS>>(
            nsteps, (int)(std::min(std::min(Ka, Kb), K) / C::BK),
            [&](int st, int j, auto in) {
                const int64_t k0 = (int64_t)j * C::BK;
                ta[st].fetch(ga, k0, !decltype(in)::value && k0 + C::BK > Ka, Ka);
                tb[st].fetch(gb, k0, !decltype(in)::value && k0 + C::BK > Kb, Kb);
            },
            [&](int st, int buf, int j, auto in) {
                const int64_t k0 = (int64_t)j * C::BK;
                ta[st].stash(smem + buf * kAs, ga, k0, !decltype(in)::value && k0 + C::BK > Ka, Ka);
                tb[st].stash(smem + 2 * kAs + buf * kBs, gb, k0, !decltype(in)::value && k0 + C::BK > Kb, Kb);
            },
            [&](int buf) {
                mma_k_g<C, decltype(edge)::value>(smem + buf * kAs, smem + 2 * kAs + buf * kBs, acc, wm, wn, lane,
                                                   nfm, nfn);
            });
    });

    const int r = lane & 15, g = lane >> 4;
    if (MODE == ABT_STORE) {
        // pipeline2 ends on a barrier after the last MFMA step, so the
        // operand buffers are free for staging the output tile
        abt_store_staged<T, C>(acc, smem, tid, wm, wn, m0, n0, M, N, Y, ldy, vec16);
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
            part[tile] = t;
        }
    }
}

// 16-byte vector access is possible when the pitch and base are aligned.
template <typename T>
static bool vec_ok(const void* p, int64_t ld) {
    constexpr int VEC = 16 / (int)sizeof(T);
    return (ld % VEC == 0) && (reinterpret_cast<uintptr_t>(p) % 16 == 0);
}

// k_atb over all (tile, split) workgroups, then k_atb_finish when the sum is split.
template <typename T, class C, int MODE, bool MIS = false>
static void run_atb(const char* label, const char* finish_label, hipStream_t st, const T* A, int64_t lda,
                    const T* B, int64_t ldb, int64_t M, int64_t N, int64_t K, int64_t chunk, int tiles_m, int tiles_n,
                    int splits, typename C::Acc* part, const T* svals, void* out, int64_t ldo, int64_t Mout) {
    {
        KernelTimer t(label, st);
        const dim3 grid(xcd_grid((int64_t)tiles_m * tiles_n * splits));
        hipLaunchKernelGGL((k_atb<T, C, MODE, MIS>), grid, dim3(C::NT), 0, st, A, lda, B, ldb, M, N, K, chunk,
                           tiles_m, tiles_n, splits, part, svals, out, ldo, Mout);
    }
    if (splits > 1) {
        KernelTimer t(finish_label, st);
        const dim3 grid((unsigned)((int64_t)tiles_m * tiles_n * C::FN * C::FM * (C::NT / 64)));
        hipLaunchKernelGGL((k_atb_finish<T, C, MODE>), grid, dim3(64 * kFinishRuns), 0, st,
                           reinterpret_cast<const typename C::AccV*>(part), M, N, tiles_m, splits, svals, out, ldo,
                           Mout);
    }
}
template <typename T, class C, int MODE, bool MIS = false, class... Args>
static void launch_abt(dim3 grid, hipStream_t st, Args... args) {
    hipLaunchKernelGGL((k_abt<T, C, MODE, MIS>), grid, dim3(C::NT), 0, st, args...);
}

// Padded copies of the operands whose pitch or base rule out 16-byte moves
// (large batches: the matrix-core tiles then read the copy many times), all
// in one launch: job q copies src (rows x cols, pitch lds) into dst
// (rows x ldd, ldd a multiple of the 16-byte chunk, dst 16-byte aligned),
// with zeros in columns cols <= j < ldd.  Each thread fills whole 16-byte
// chunks of dst from the two aligned 16-byte chunks of the source that cover
// them (funnel-shifted), so loads and stores are full 16-byte moves.
template <typename T>
struct StageJobs {
    const T* src[3];
    T* dst[3];
    int64_t rows[3], cols[3], lds[3];
    int cpr[3];              // 16-byte chunks per destination row
    int64_t chunks[3];       // chunks of job q
    unsigned bend[3];        // workgroups up to and including job q
    int n;
};

template <typename T, typename I>
__global__ __launch_bounds__(256) void k_pitch_copy(StageJobs<T> J) {
    constexpr int VEC = 16 / (int)sizeof(T);
    typedef T vec_t __attribute__((ext_vector_type(VEC)));
    // the job is uniform over the workgroup: its fields come from scalar loads
    const unsigned bid = blockIdx.x;
    const int q = bid < J.bend[0] ? 0 : (bid < J.bend[1] ? 1 : 2);
    const unsigned b0 = q == 0 ? 0u : J.bend[q - 1];
    const I nb = (I)(J.bend[q] - b0);
    const I total = (I)J.chunks[q];
    const I cpr = (I)J.cpr[q];
    const T* src = J.src[q];
    T* dst = J.dst[q];
    const int64_t lds = J.lds[q], cols = J.cols[q];
    const T* last = src + (J.rows[q] - 1) * lds + (cols - 1);
    for (I c = (I)(bid - b0) * 256 + threadIdx.x; c < total; c += nb * 256) {
        const I i = c / cpr;
        const int64_t j0 = (int64_t)(c - i * cpr) * VEC;
        MisChunk<T> mc;   // chunks past the row's end start at its last element (their values are zeroed)
        mc.fetch(src + (int64_t)i * lds + (j0 < cols ? j0 : cols - 1), last);
        vec_t w = mc.template value<vec_t>();
#pragma unroll
        for (int v = 0; v < VEC; ++v)
            if (j0 + v >= cols) w[v] = T(0);
        *reinterpret_cast<vec_t*>(dst + (int64_t)c * VEC) = w;
    }
}

// --------------------------------------------------------- streaming path --
// Batches of at most NB = 8 columns, two launches.
//
// Phase 1 (k_p1_thin): workgroup (jg, sp) of 8 waves owns columns
// [64 jg, 64 jg + 64) of V and a chunk of rows of V and X.  Lane j of every
// wave accumulates column j over the wave's contiguous share of the chunk, in
// batches of RW rows whose loads are all issued before the first product
// (V element by element along its rows, which a wave reads as whole 128-byte
// segments whatever the row pitch; the batch's X rows, contiguous in memory,
// by one coalesced load per lane into the wave's own LDS rows, from which
// every lane reads them).  The waves are added in wave order and the
// workgroup writes its partial.  (A last-workgroup finish inside this kernel
// needs a device-scope release per workgroup, which on this chip writes back
// the L2 of its XCD each time and measured slower than a second launch.)
constexpr int kThinWaves = 8;
constexpr int kThinRows = 32;                    // rows per wave and batch

template <typename T, int NB>
__global__ __launch_bounds__(64 * kThinWaves) void k_p1_thin(
    const T* __restrict__ V, const T* __restrict__ X, typename PrecTraits<T>::acc* __restrict__ part,
    int64_t n, int64_t k, int64_t b, int64_t chunk, int splits) {
    using Acc = typename PrecTraits<T>::acc;
    constexpr int W = kThinWaves, RW = kThinRows;
    __shared__ Acc red[W][64][NB];
    __shared__ Acc xs[W][RW * NB];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int jg = blockIdx.x, sp = blockIdx.y;
    const int64_t j = (int64_t)jg * 64 + lane;
    const int64_t jc = j < k ? j : k - 1;        // clamped column: loads stay inside V
    const int64_t c0 = (int64_t)sp * chunk;
    const int64_t c1 = (c0 + chunk < n) ? c0 + chunk : n;
    const int64_t q = (c1 - c0 + W - 1) / W;     // rows of this wave's share
    const int64_t i0 = c0 + wave * q;
    const int64_t i1 = (i0 + q < c1) ? i0 + q : c1;

    Acc acc[NB];
#pragma unroll
    for (int c = 0; c < NB; ++c) acc[c] = 0;
    for (int64_t ib = i0; ib < i1; ib += RW) {
        const int rows = (int)((i1 - ib < RW) ? i1 - ib : RW);
        T v[RW];
#pragma unroll
        for (int r = 0; r < RW; ++r) v[r] = V[(ib + (r < rows ? r : rows - 1)) * k + jc];
        // the batch's X values, rows ib .. ib + rows - 1 (rows * b contiguous values)
        constexpr int XL = (RW * NB + 63) / 64;
        Acc xv[XL];
#pragma unroll
        for (int t = 0; t < XL; ++t) {
            const int e = t * 64 + lane;                 // (row, column) = (e / NB, e % NB)
            const int r = e / NB, c = e - r * NB;
            xv[t] = (r < rows && c < b) ? to_acc(X[(ib + r) * b + c]) : Acc(0);
        }
#pragma unroll
        for (int t = 0; t < XL; ++t)
            if (t * 64 + lane < RW * NB) xs[wave][t * 64 + lane] = xv[t];
        __builtin_amdgcn_wave_barrier();                 // LDS writes of this wave before its reads
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            if (r < rows) {   // predicated, so v[] stays in registers
                const Acc vij = to_acc(v[r]);
#pragma unroll
                for (int c = 0; c < NB; ++c) acc[c] += vij * xs[wave][r * NB + c];
            }
        }
        __builtin_amdgcn_wave_barrier();                 // reads done before the next batch's writes
    }
#pragma unroll
    for (int c = 0; c < NB; ++c) red[wave][lane][c] = acc[c];
    __syncthreads();
    if (wave == 0) {
        Acc* dst = part + (((int64_t)jg * splits + sp) * 64 + lane) * NB;
#pragma unroll
        for (int c = 0; c < NB; ++c) {
            Acc t = red[0][lane][c];
#pragma unroll
            for (int w = 1; w < W; ++w) t += red[w][lane][c];
            dst[c] = t;
        }
    }
}

// T'[j][c] = s_j * (sum of the chunk partials of (j, c) in chunk order):
// one wave per output (j, c) of T'^T, including the zero rows j in [k, ldt),
// lane l adding the partials l, l + 64, ... then a fixed butterfly.  Used
// when the batch is wider than the phase-2 kernel folds in itself.
template <typename T, int NB>
__global__ __launch_bounds__(256) void k_p1_thin_finish(
    const typename PrecTraits<T>::acc* __restrict__ part, const T* __restrict__ s, T* __restrict__ Tt,
    int64_t ldt, int64_t k, int64_t b, int splits) {
    using Acc = typename PrecTraits<T>::acc;
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= ldt * NB) return;
    const int64_t jj = w / NB;
    const int c = (int)(w - jj * NB);
    if (c >= b) return;
    Acc sum = 0;
    if (jj < k) {
        const int64_t jg = jj / 64, jl = jj - jg * 64;
        const Acc* src = part + (jg * splits * 64 + jl) * NB + c;
        for (int t = lane; t < splits; t += 64) sum += src[(int64_t)t * 64 * NB];
        sum = wave_sum(sum);
    }
    if (lane == 0) {
        const Acc sj = (jj < k) ? to_acc(s[jj]) : Acc(0);
        Tt[(int64_t)c * ldt + jj] = to_storage<T>(sj * sum);
    }
}

// Phase 2 (k_p2_thin): every wave owns RPW rows of U; lanes stride over j.
// The U loads of the first batch of column groups are issued first; then
// T' (k x NB) is formed in LDS, either from T'^T or (FOLD) by adding the
// chunk partials of phase 1 in chunk order and scaling by s -- the same sum
// and order as k_p1_thin_finish, done by every workgroup instead of by a
// third launch; then each lane multiplies its U values by T' from LDS, and a
// fixed butterfly over the wave gives each output.
template <typename T, int NB, bool FOLD>
__global__ __launch_bounds__(256) void k_p2_thin(
    const T* __restrict__ U, const T* __restrict__ Tt, int64_t ldt, const typename PrecTraits<T>::acc* __restrict__ part,
    const T* __restrict__ s, int splits, T* __restrict__ Y, int64_t m, int64_t k, int64_t b) {
    using Acc = typename PrecTraits<T>::acc;
    constexpr int RPW = 4, JB = 4;
    extern __shared__ double4_t smem_v[];
    Acc* ts = reinterpret_cast<Acc*>(smem_v);    // T'[j][c], k x NB
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t row0 = ((int64_t)blockIdx.x * 4 + wave) * RPW;
    int64_t rows[RPW];
#pragma unroll
    for (int r = 0; r < RPW; ++r) rows[r] = (row0 + r < m) ? row0 + r : m - 1;   // clamped: loads stay inside U
    T u[RPW][JB];
    auto load_u = [&](int64_t jb) {
#pragma unroll
        for (int t = 0; t < JB; ++t) {
            const int64_t jj = jb + 64 * t + lane;
            const int64_t jc = jj < k ? jj : k - 1;
#pragma unroll
            for (int r = 0; r < RPW; ++r) u[r][t] = U[rows[r] * k + jc];
        }
    };
    load_u(0);
    for (int64_t idx = tid; idx < k * NB; idx += 256) {
        const int64_t jj = idx / NB;
        const int c = (int)(idx - jj * NB);
        Acc val = 0;
        if (c < b) {
            if constexpr (FOLD) {
                const int64_t jg = jj / 64, jl = jj - jg * 64;
                const Acc* src = part + (jg * splits * 64 + jl) * NB + c;
                Acc sum = 0;
                for (int t = 0; t < splits; t += 16) {   // 16 loads in flight, added in chunk order
                    Acc pv[16];
#pragma unroll
                    for (int u = 0; u < 16; ++u) pv[u] = (t + u < splits) ? src[(int64_t)(t + u) * 64 * NB] : Acc(0);
#pragma unroll
                    for (int u = 0; u < 16; ++u) sum += pv[u];
                }
                val = to_acc(to_storage<T>(to_acc(s[jj]) * sum));   // T' as stored: rounded to T
            } else {
                val = to_acc(Tt[(int64_t)c * ldt + jj]);
            }
        }
        ts[idx] = val;
    }
    __syncthreads();
    Acc acc[RPW][NB];
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int c = 0; c < NB; ++c) acc[r][c] = 0;
    for (int64_t jb = 0; jb < k; jb += 64 * JB) {
        if (jb > 0) load_u(jb);
#pragma unroll
        for (int t = 0; t < JB; ++t) {
            const int64_t jj = jb + 64 * t + lane;
            if (jj < k) {
#pragma unroll
                for (int r = 0; r < RPW; ++r)
#pragma unroll
                    for (int c = 0; c < NB; ++c) acc[r][c] += to_acc(u[r][t]) * ts[jj * NB + c];
            }
        }
    }
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int c = 0; c < NB; ++c) acc[r][c] = wave_sum(acc[r][c]);
    // lane r * NB + c writes output (row0 + r, c)
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int c = 0; c < NB; ++c)
            if (lane == r * NB + c && row0 + r < m && c < b) Y[(row0 + r) * b + c] = to_storage<T>(acc[r][c]);
}

// ------------------------------------------------------------------- host --
static constexpr int kStreamMaxBatch = 8;
static constexpr int kStreamRowsTarget = kThinWaves * kThinRows;   // rows of V per phase-1 chunk
static constexpr int kStreamMaxSplits = 32;
static constexpr int kStreamFoldBatch = 2;       // phase 2 adds the chunk partials itself up to this batch

static constexpr size_t kInPlaceBytes = (size_t)16 << 20;  // shifted-load budget of an in-place factor
static constexpr int64_t kBigTarget = 512;       // phase-1 workgroups aimed for (128 x 128 tiles)
static constexpr int64_t kSmallTarget = 1024;    // same for 64 x 64 tiles
static constexpr int64_t kFewTiles = 16;         // phase-1 outputs of fewer tiles than this ...
static constexpr int64_t kFewTarget = 256;       // ... aim for this many workgroups

// LRC_APPLY_TILE=64 or 128 pins the MFMA tile edge of both phases (tuning aid).
static int forced_tile() {
    static const int t = [] {
        const char* e = std::getenv("LRC_APPLY_TILE");
        const int v = e ? std::atoi(e) : 0;
        return (v == 64 || v == 128) ? v : 0;
    }();
    return t;
}

static bool needs_stage(const void* p, int64_t ld, int prec) {
    const int64_t vec = 16 / (int64_t)elem_bytes(prec);
    return (ld % vec != 0) || (reinterpret_cast<uintptr_t>(p) % 16 != 0);
}

// Tile edges and K step of the matrix-core configurations, for the plan (the
// grids and the split-K partial buffers are sized from the same constants
// the kernels are compiled with).
struct TileDims {
    int bm, bn, bk;
};
template <class C>
static TileDims dims_of() {
    return TileDims{C::BM, C::BN, C::BK};
}
template <typename T> struct PrecCode;
template <> struct PrecCode<double> { static constexpr int value = P64; };
template <> struct PrecCode<float> { static constexpr int value = P32; };
template <> struct PrecCode<half_t> { static constexpr int value = P16; };
static TileDims cfg_dims(int prec, bool big) {
    if (prec == P64) return big ? dims_of<BigCfg<double>::C>() : dims_of<SmallCfg<double>::C>();
    if (prec == P32) return big ? dims_of<BigCfg<float>::C>() : dims_of<SmallCfg<float>::C>();
    return big ? dims_of<BigCfg<half_t>::C>() : dims_of<SmallCfg<half_t>::C>();
}

ApplyPlan plan_apply(int64_t m, int64_t n, int64_t k, int64_t b, int prec, int path, const void* U,
                     const void* V, const void* X) {
    ApplyPlan p{};
    if (path != 1 && path != 2) path = (b <= kStreamMaxBatch) ? 1 : 2;
    if (path == 1 && b > kStreamMaxBatch) path = 2;
    // the streaming phase 2 keeps T' (k x batch, accumulation type) in 64 KB
    // of LDS: ranks whose T' does not fit take the matrix-core path
    if (path == 1) {
        const int64_t nb = (b <= 1) ? 1 : (b <= 2) ? 2 : (b <= 4) ? 4 : 8;
        if (k * nb * ((prec == P64) ? 8 : 4) > 65536) path = 2;
    }

    p.path = path;
    // Rows of T'^T and of staged factor copies: on the matrix-core path a
    // whole number of 64-byte K steps (32 halves, 16 floats, 8 doubles), so
    // that each step's slice of a row is one aligned 64-byte segment rather
    // than one that straddles two cache lines; the K steps are as many.
    p.Kp = round_up(k, path == 2 ? 64 / (int64_t)elem_bytes(prec) : 8);
    const size_t acc_b = (prec == P64) ? 8 : 4;
    if (path == 1) {
        p.tiles_m = (int)((k + 63) / 64);
        p.tiles_n = 1;
        int64_t splits = (n + kStreamRowsTarget - 1) / kStreamRowsTarget;
        if (splits > kStreamMaxSplits) splits = kStreamMaxSplits;
        if (splits < 1) splits = 1;
        p.chunk = (n + splits - 1) / splits;
        p.splits = (int)((n + p.chunk - 1) / p.chunk);
        const int nb = (b <= 1) ? 1 : (b <= 2) ? 2 : (b <= 4) ? 4 : 8;
        p.part_bytes = (size_t)p.tiles_m * p.splits * 64 * nb * acc_b;
    } else {
        // phase 1: C = V^T X is k x b, summed over n.  Big tiles only where they
        // pad the k rows no more than the small ones (k + 1 = 257: three
        // 128-row tiles hold 384 rows, five 64-row tiles 320; measured 279 ->
        // 246 us FP32, 70 -> 56 us FP16 at n = 8192, b = 4096)
        {
            const TileDims db = cfg_dims(prec, true), ds = cfg_dims(prec, false);
            const int64_t pad_b = round_up(k, db.bm) - k, pad_s = round_up(k, ds.bm) - k;
            p.big1 = (k >= 128 && b >= 128 && pad_b <= pad_s) ? 1 : 0;
        }
        if (forced_tile()) p.big1 = forced_tile() == 128;
        const TileDims d1 = cfg_dims(prec, p.big1);
        const int BK = d1.bk;
        p.tiles_m = (int)((k + d1.bm - 1) / d1.bm);
        p.tiles_n = (int)((b + d1.bn - 1) / d1.bn);
        const int64_t base = (int64_t)p.tiles_m * p.tiles_n;
        // Outputs of many tiles: about kBigTarget / kSmallTarget workgroups
        // with at least 16 K steps per split (more splits only lengthen the
        // finish's sums).  Outputs of a few tiles (small k x batch): about one
        // workgroup per compute unit with at least 4 K steps each, so that
        // the few tiles still spread over the chip; the finish adds the
        // partials in eight parallel runs.
        const bool few = base < kFewTiles;
        const int64_t target = few ? kFewTarget : p.big1 ? kBigTarget : kSmallTarget;
        int64_t splits = (target + base - 1) / base;
        int64_t max_splits = n / ((few ? 4 : 16) * BK);
        if (max_splits < 1) max_splits = 1;
        if (splits > max_splits) splits = max_splits;
        if (splits < 1) splits = 1;
        p.chunk = round_up((n + splits - 1) / splits, BK);
        p.splits = (int)((n + p.chunk - 1) / p.chunk);
        p.part_bytes = (p.splits > 1) ? (size_t)base * p.splits * d1.bm * d1.bn * acc_b : 0;
        // phase 2: Y = U T' is m x b
        const int64_t big_tiles = ((m + 127) / 128) * ((b + 127) / 128);
        p.big2 = (m >= 128 && b >= 128 && big_tiles >= 256) ? 1 : 0;
        if (forced_tile()) p.big2 = forced_tile() == 128;
    }
    p.mid_bytes = (size_t)b * p.Kp * elem_bytes(prec);
    if (path == 2) {
        // A misaligned factor is read in place (two aligned loads and a shift
        // per chunk) when the shifted loads add up to little: the factor's
        // bytes times the column tiles that read it at most kInPlaceBytes
        // (a single column tile reads each element once).  Then the copy's
        // extra launch costs more than the shifts; otherwise the factor is
        // copied to a padded pitch once per call (measured at 8192 x 8192,
        // batch 4096: in place, phases 1 and 2 each lose 15-25 %, more than
        // the copy costs).  A misaligned X is always copied.
        const TileDims d1 = cfg_dims(prec, p.big1), d2 = cfg_dims(prec, p.big2);
        const size_t e = elem_bytes(prec);
        const bool u_bad = needs_stage(U, k, prec), v_bad = needs_stage(V, k, prec);
        const size_t reads1 = (size_t)((b + d1.bn - 1) / d1.bn), reads2 = (size_t)((b + d2.bn - 1) / d2.bn);
        p.mis1 = (v_bad && (reads1 <= 1 || (size_t)n * k * e * reads1 <= kInPlaceBytes)) ? 1 : 0;
        p.mis2 = (u_bad && (reads2 <= 1 || (size_t)m * k * e * reads2 <= kInPlaceBytes)) ? 1 : 0;
        p.stage_u = (u_bad && !p.mis2) ? 1 : 0;
        p.stage_v = (v_bad && !p.mis1) ? 1 : 0;
        p.stage_x = needs_stage(X, b, prec) ? 1 : 0;
        p.ldx = round_up(b, 8);
        p.stage_bytes = (p.stage_u ? round_up((size_t)m * p.Kp * e, 256) : 0) +
                        (p.stage_v ? round_up((size_t)n * p.Kp * e, 256) : 0) +
                        (p.stage_x ? round_up((size_t)n * p.ldx * e, 256) : 0);
    }
    return p;
}

size_t apply_workspace_bytes(const ApplyPlan& p) {
    return round_up(p.part_bytes, 256) + round_up(p.mid_bytes, 256) + p.stage_bytes;
}

template <typename T> static const char* p1_stream_label();
template <typename T> static const char* p2_stream_label();
template <typename T> static const char* p1_mfma_label();
template <typename T> static const char* p2_mfma_label();
template <typename T> static const char* p1_finish_label();
#define LRC_LABELS(T, S)                                                          \
    template <> const char* p1_stream_label<T>() { return "apply_p1_stream_" S; } \
    template <> const char* p2_stream_label<T>() { return "apply_p2_stream_" S; } \
    template <> const char* p1_mfma_label<T>() { return "apply_p1_mfma_" S; }     \
    template <> const char* p2_mfma_label<T>() { return "apply_p2_mfma_" S; }     \
    template <> const char* p1_finish_label<T>() { return "apply_p1_finish_" S; }
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
    if (ws.overrun || !Tt) return hipErrorOutOfMemory;
    const int64_t ldt = p.Kp;
    if (p.path == 1) {
        const int nb = b <= 1 ? 1 : b <= 2 ? 2 : b <= 4 ? 4 : 8;
        const bool fold = b <= kStreamFoldBatch;
        const dim3 g1(p.tiles_m, p.splits);
        {
            KernelTimer t1(p1_stream_label<T>(), stream);
#define LRC_P1S(NB)                                                                                            \
    hipLaunchKernelGGL((k_p1_thin<T, NB>), g1, dim3(64 * kThinWaves), 0, stream, V, X, part, n, k, b, p.chunk, \
                       p.splits)
            if (nb == 1) LRC_P1S(1); else if (nb == 2) LRC_P1S(2); else if (nb == 4) LRC_P1S(4); else LRC_P1S(8);
#undef LRC_P1S
        }
        if (!fold) {
            KernelTimer tf(p1_finish_label<T>(), stream);
            const dim3 gf((unsigned)((ldt * nb + 3) / 4));
#define LRC_P1F(NB) \
    hipLaunchKernelGGL((k_p1_thin_finish<T, NB>), gf, dim3(256), 0, stream, part, s, Tt, ldt, k, b, p.splits)
            if (nb == 4) LRC_P1F(4); else LRC_P1F(8);
#undef LRC_P1F
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        const int64_t rows_per_wg = 16;
        const dim3 g2((unsigned)((m + rows_per_wg - 1) / rows_per_wg));
        const size_t lds = (size_t)k * nb * sizeof(Acc);
        KernelTimer t2(p2_stream_label<T>(), stream);
#define LRC_P2S(NB, F)                                                                                       \
    hipLaunchKernelGGL((k_p2_thin<T, NB, F>), g2, dim3(256), lds, stream, U, Tt, ldt, part, s, p.splits, Y, m, k, \
                       b)
        if (nb == 1) LRC_P2S(1, true); else if (nb == 2) LRC_P2S(2, true); else if (nb == 4) LRC_P2S(4, false);
        else LRC_P2S(8, false);
#undef LRC_P2S
        return hipGetLastError();
    }
    // operands whose pitch or base rule out 16-byte moves, unless read in place
    const T *Ug = U, *Vg = V, *Xg = X;
    int64_t ldu = k, ldv = k, ldx = b;
    if (p.stage_u || p.stage_v || p.stage_x) {
        StageJobs<T> J{};
        auto add = [&](const T* src, int64_t rows, int64_t cols, int64_t ldd) -> T* {
            T* d = static_cast<T*>(ws.take((size_t)rows * ldd * sizeof(T)));
            if (!d) return nullptr;
            const int q = J.n++;
            J.src[q] = src;
            J.dst[q] = d;
            J.rows[q] = rows;
            J.cols[q] = cols;
            J.lds[q] = cols;
            J.cpr[q] = (int)(ldd / (16 / (int64_t)sizeof(T)));
            J.chunks[q] = rows * J.cpr[q];
            int64_t nb = (J.chunks[q] + 255) / 256;
            if (nb > 4096) nb = 4096;
            J.bend[q] = (q ? J.bend[q - 1] : 0u) + (unsigned)nb;
            return d;
        };
        if (p.stage_u) {
            T* d = add(U, m, k, p.Kp);
            if (!d) return hipErrorOutOfMemory;
            Ug = d;
            ldu = p.Kp;
        }
        if (p.stage_v) {
            T* d = add(V, n, k, p.Kp);
            if (!d) return hipErrorOutOfMemory;
            Vg = d;
            ldv = p.Kp;
        }
        if (p.stage_x) {
            T* d = add(X, n, b, p.ldx);
            if (!d) return hipErrorOutOfMemory;
            Xg = d;
            ldx = p.ldx;
        }
        KernelTimer ts("apply_stage", stream);
        const dim3 grid(J.bend[J.n - 1]);
        bool small = true;
        for (int q = 0; q < J.n; ++q) small = small && J.chunks[q] < ((int64_t)1 << 31);
        if (small)
            hipLaunchKernelGGL((k_pitch_copy<T, uint32_t>), grid, dim3(256), 0, stream, J);
        else
            hipLaunchKernelGGL((k_pitch_copy<T, int64_t>), grid, dim3(256), 0, stream, J);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    using Big = typename BigCfg<T>::C;
    using Small = typename SmallCfg<T>::C;
    const char *l1 = p1_mfma_label<T>(), *lf = p1_finish_label<T>();
#define LRC_P1(CFG, MISV)                                                                                        \
    run_atb<T, CFG, ATB_APPLY, MISV>(l1, lf, stream, Vg, ldv, Xg, ldx, k, b, n, p.chunk, p.tiles_m, p.tiles_n,     \
                                     p.splits, part, s, (void*)Tt, ldt, ldt)
    if (p.big1) {
        if (p.mis1) LRC_P1(Big, true); else LRC_P1(Big, false);
    } else {
        if (p.mis1) LRC_P1(Small, true); else LRC_P1(Small, false);
    }
#undef LRC_P1
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    KernelTimer t2(p2_mfma_label<T>(), stream);
    const int vec16 = vec_ok<T>(Y, b) ? 1 : 0;
    const TileDims d2 = cfg_dims(PrecCode<T>::value, p.big2);
    const int tm = (int)((m + d2.bm - 1) / d2.bm), tn = (int)((b + d2.bn - 1) / d2.bn);
    const dim3 g2(xcd_grid(AbtOrder(tm, tn).total));
#define LRC_P2(CFG, MISV)                                                                                       \
    launch_abt<T, CFG, ABT_STORE, MISV>(g2, stream, Ug, ldu, m, k, (const T*)Tt, ldt, b, ldt, ldt, tm, tn, Y, b,     \
                                        vec16, (const double*)nullptr, (int64_t)0, (double*)nullptr)
    if (p.big2) {
        if (p.mis2) LRC_P2(Big, true); else LRC_P2(Big, false);
    } else {
        if (p.mis2) LRC_P2(Small, true); else LRC_P2(Small, false);
    }
#undef LRC_P2
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

// Split of the Gram's row range: about 1536 workgroups of 64 x 64 tiles
// (measured on the 8192 x 514 factor blocks: 1024 leaves the compute units
// unevenly loaded, beyond 2048 the partial tiles cost more than they save).
static void gram_plan(int64_t rows, int64_t cols, int* tiles, int* splits, int64_t* chunk) {
    static_assert(GramC::BM == GramC::BN, "square Gram tiles");
    const int t = (int)((cols + GramC::BM - 1) / GramC::BM);
    const int64_t base = (int64_t)t * t;
    int64_t sp = (1536 + base - 1) / base;
    // at least 64 rows per split, 256 for Grams of at most 2 x 2 tiles
    // (those would otherwise spend more on their partial tiles than on the
    // product)
    int64_t mx = rows / (base <= 4 ? 256 : 64);
    if (mx < 1) mx = 1;
    if (sp > mx) sp = mx;
    if (sp < 1) sp = 1;
    *chunk = round_up((rows + sp - 1) / sp, GramC::BK);
    *splits = (int)((rows + *chunk - 1) / *chunk);
    *tiles = t;
}

size_t gram_workspace_bytes(int64_t rows, int64_t cols) {
    int t, sp;
    int64_t ch;
    gram_plan(rows, cols, &t, &sp, &ch);
    return (size_t)t * t * sp * GramC::BM * GramC::BN * sizeof(double);
}

hipError_t launch_gram(const double* P, int64_t rows, int64_t cols, double* G, Workspace& ws,
                       hipStream_t stream) {
    int t, sp;
    int64_t ch;
    gram_plan(rows, cols, &t, &sp, &ch);
    double* part = static_cast<double*>(ws.take(gram_workspace_bytes(rows, cols)));
    if (ws.overrun) return hipErrorOutOfMemory;
    if (!vec_ok<double>(P, cols)) return hipErrorInvalidValue;   // the factor builders keep 2r columns
    run_atb<double, GramC, ATB_GRAM>("cert_gram_f64", "cert_gram_finish_f64", stream, P, cols, P, cols, cols, cols,
                                     rows, ch, t, t, sp, part, (const double*)nullptr, (void*)G, cols, cols);
    return hipGetLastError();
}

size_t err_workspace_bytes(int64_t m, int64_t n) {
    return (size_t)((m + GramC::BM - 1) / GramC::BM) * ((n + GramC::BN - 1) / GramC::BN) * sizeof(double);
}

hipError_t launch_err_dense(const double* A, const double* W, const double* Vw, int64_t m, int64_t n,
                            int64_t r, int64_t ldw, double* part, int64_t* nparts, hipStream_t stream) {
    const int tm = (int)((m + GramC::BM - 1) / GramC::BM), tn = (int)((n + GramC::BN - 1) / GramC::BN);
    *nparts = (int64_t)tm * tn;
    const int64_t K = round_up(r, GramC::BK);
    if (!vec_ok<double>(W, ldw) || !vec_ok<double>(Vw, ldw)) return hipErrorInvalidValue;
    KernelTimer tm_("cert_err_dense_f64", stream);
    launch_abt<double, GramC, ABT_ERR>(dim3(xcd_grid(AbtOrder(tm, tn).total)), stream, W, ldw, m, r, Vw, ldw, n, r, K, tm, tn,
                                       (double*)nullptr, (int64_t)0, 0, A, n, part);
    return hipGetLastError();
}

// ------------------------------------------------- factorization GEMMs (FP64)
// Split-K partial tiles of C[m][n] = sum_{k in split} A[m][k] B[n][k] (both
// sources K-contiguous, 16-byte aligned with even pitches), in the layout of
// k_atb's partials (tile = n tile * tiles_m + m tile): k_atb_finish in
// ATB_APPLY mode sums them in split order and stores C transposed.
template <class C>
__global__ __launch_bounds__(C::NT) void k_abt_part(const double* __restrict__ Asrc, int64_t lda, int64_t M,
                                                    const double* __restrict__ Bsrc, int64_t ldb, int64_t N,
                                                    int64_t K, int64_t chunk, int tiles_m, int tiles_n, int splits,
                                                    double* __restrict__ part) {
    using AccV = typename C::AccV;
    constexpr int kAs = C::BM * C::LDK, kBs = C::BN * C::LDK;
    __shared__ alignas(16) double smem[2 * kAs + 2 * kBs];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave / C::WN, wn = wave % C::WN;
    const int64_t ntile = (int64_t)tiles_m * tiles_n;
    const int64_t lt = xcd_tile(ntile * splits);
    if (lt >= ntile * splits) return;
    const int64_t tile = lt % ntile;
    const int sp = (int)(lt / ntile);
    const int64_t m0 = (tile % tiles_m) * C::BM, n0 = (tile / tiles_m) * C::BN;
    const int nfm = live_frags<C::FM>(m0 + wm * C::WTM, M), nfn = live_frags<C::FN>(n0 + wn * C::WTN, N);
    const int64_t kbeg = (int64_t)sp * chunk;
    const int64_t kend = (kbeg + chunk < K) ? kbeg + chunk : K;
    AccV acc[C::FN][C::FM];
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) acc[fn][fm] = zero_accv<AccV>();
    using TA = KTile<C, C::BM, double>;
    using TB = KTile<C, C::BN, double>;
    const typename TA::Geo ga = TA::geo(Asrc, lda, m0, M, tid);
    const typename TB::Geo gb = TB::geo(Bsrc, ldb, n0, N, tid);
    TA ta[2];
    TB tb[2];
    const int nsteps = (int)((kend - kbeg + C::BK - 1) / C::BK);
    by_edge(nfm == C::FM && nfn == C::FN, [&](auto edge) {
        // The edge-free inner loop measured no faster for these split-K tiles.
        pipeline2<false>(
            nsteps, (int)((kend - kbeg) / C::BK),
            [&](int st, int j, auto in) {
                const int64_t k0 = kbeg + (int64_t)j * C::BK;
                const bool pk = !decltype(in)::value && k0 + C::BK > kend;
                ta[st].fetch(ga, k0, pk, kend);
                tb[st].fetch(gb, k0, pk, kend);
            },
            [&](int st, int buf, int j, auto in) {
                const int64_t k0 = kbeg + (int64_t)j * C::BK;
                const bool pk = !decltype(in)::value && k0 + C::BK > kend;
                ta[st].stash(smem + buf * kAs, ga, k0, pk, kend);
                tb[st].stash(smem + 2 * kAs + buf * kBs, gb, k0, pk, kend);
            },
            [&](int buf) {
                mma_k_g<C, decltype(edge)::value>(smem + buf * kAs, smem + 2 * kAs + buf * kBs, acc, wm, wn, lane,
                                                   nfm, nfn);
            });
    });
    constexpr int NF = C::FN * C::FM;
    AccV* mine = reinterpret_cast<AccV*>(part) + ((tile * splits + sp) * NF) * C::NT + tid;
#pragma unroll
    for (int fn = 0; fn < C::FN; ++fn)
#pragma unroll
        for (int fm = 0; fm < C::FM; ++fm) mine[(fn * C::FM + fm) * C::NT] = acc[fn][fm];
}

// Splits of a K range over `tiles` output tiles: about 1536 workgroups, at
// least 256 K values per split (chunk a multiple of the K step).
static void split_plan(int64_t tiles, int64_t K, int* splits, int64_t* chunk) {
    int64_t sp = (1536 + tiles - 1) / tiles;
    int64_t mx = K / 256;
    if (mx < 1) mx = 1;
    if (sp > mx) sp = mx;
    if (sp < 1) sp = 1;
    *chunk = round_up((K + sp - 1) / sp, GramC::BK);
    *splits = (int)((K + *chunk - 1) / *chunk);
}

static int64_t tiles_of(int64_t n, int b) { return (n + b - 1) / b; }

// At most 96 rows of W (the factorization's sketches and small factors) take
// one 96-row tile, three fragments per wave (75 test vectors leave 21 of 96
// rows idle instead of 53 of 128); wider W takes the 64 x 64 tiles.
using NarrowC = Cfg<double, 96, 64, 16, 2, 2>;

template <class C>
static size_t gemm_nt_bytes(int64_t nw, int64_t rows, int64_t K) {
    const int64_t tiles = tiles_of(nw, C::BM) * tiles_of(rows, C::BN);
    int sp;
    int64_t ch;
    split_plan(tiles, K, &sp, &ch);
    return (size_t)tiles * sp * C::BM * C::BN * sizeof(double);
}

size_t gemm_nt_workspace_bytes(int64_t nw, int64_t rows, int64_t K) {
    return nw <= NarrowC::BM ? gemm_nt_bytes<NarrowC>(nw, rows, K) : gemm_nt_bytes<GramC>(nw, rows, K);
}

template <class C>
static hipError_t gemm_nt_typed(const double* W, int64_t ldw, int64_t nw, const double* A, int64_t lda, int64_t rows,
                                int64_t K, const double* svals, double* out, int64_t ldo, int64_t mout, Workspace& ws,
                                hipStream_t stream, const char* label) {
    const int tm = (int)tiles_of(nw, C::BM), tn = (int)tiles_of(rows, C::BN);
    if (!vec_ok<double>(W, ldw) || !vec_ok<double>(A, lda) || mout < nw || mout > (int64_t)tm * C::BM)
        return hipErrorInvalidValue;
    int sp;
    int64_t ch;
    split_plan((int64_t)tm * tn, K, &sp, &ch);
    double* part = static_cast<double*>(ws.take(gemm_nt_bytes<C>(nw, rows, K)));
    if (ws.overrun) return hipErrorOutOfMemory;
    KernelTimer t(label, stream);
    hipLaunchKernelGGL(k_abt_part<C>, dim3(xcd_grid((int64_t)tm * tn * sp)), dim3(C::NT), 0, stream, W, ldw, nw, A,
                       lda, rows, K, ch, tm, tn, sp, part);
    hipLaunchKernelGGL((k_atb_finish<double, C, ATB_APPLY>),
                       dim3((unsigned)((int64_t)tm * tn * C::FN * C::FM * (C::NT / 64))), dim3(64 * kFinishRuns), 0,
                       stream, reinterpret_cast<const typename C::AccV*>(part), nw, rows, tm, sp, svals, (void*)out,
                       ldo, mout);
    return hipGetLastError();
}

hipError_t launch_gemm_nt(const double* W, int64_t ldw, int64_t nw, const double* A, int64_t lda, int64_t rows,
                          int64_t K, const double* svals, double* out, int64_t ldo, int64_t mout, Workspace& ws,
                          hipStream_t stream, const char* label) {
    if (nw <= NarrowC::BM)
        return gemm_nt_typed<NarrowC>(W, ldw, nw, A, lda, rows, K, svals, out, ldo, mout, ws, stream, label);
    return gemm_nt_typed<GramC>(W, ldw, nw, A, lda, rows, K, svals, out, ldo, mout, ws, stream, label);
}

size_t gemm_tn_workspace_bytes(int64_t nq, int64_t cols, int64_t K) {
    const int64_t tiles = tiles_of(nq, GramC::BM) * tiles_of(cols, GramC::BN);
    int sp;
    int64_t ch;
    split_plan(tiles, K, &sp, &ch);
    return sp > 1 ? (size_t)tiles * sp * GramC::BM * GramC::BN * sizeof(double) : 0;
}

hipError_t launch_gemm_tn(const double* Q, int64_t ldq, int64_t nq, const double* A, int64_t lda, int64_t cols,
                          int64_t K, double* out, int64_t ldo, int64_t mout, Workspace& ws, hipStream_t stream,
                          const char* label, const char* finish_label) {
    const int tm = (int)tiles_of(nq, GramC::BM), tn = (int)tiles_of(cols, GramC::BN);
    if (!vec_ok<double>(Q, ldq) || !vec_ok<double>(A, lda) || mout < nq || mout > (int64_t)tm * GramC::BM)
        return hipErrorInvalidValue;
    int sp;
    int64_t ch;
    split_plan((int64_t)tm * tn, K, &sp, &ch);
    double* part = nullptr;
    if (sp > 1) {
        part = static_cast<double*>(ws.take(gemm_tn_workspace_bytes(nq, cols, K)));
        if (ws.overrun) return hipErrorOutOfMemory;
    }
    run_atb<double, GramC, ATB_APPLY>(label, finish_label, stream, Q, ldq, A, lda, nq, cols, K, ch, tm, tn, sp, part,
                                      (const double*)nullptr, (void*)out, ldo, mout);
    return hipGetLastError();
}

}  // namespace lrc

// Fused Tensor-Train reconstruction for gfx950 (Sec. 5.1; Sec. 7.5
// eq. gpu_tt_reconstruction).
//
// The paper contracts the cores left to right, B_l = Z_{l-1} K_l, through
// preallocated buffers in global memory.  Here the dense tensor, viewed as a
// matrix with rows (i_1..i_{d-1}) and columns i_d, is cut into blocks of
// P rows; one workgroup produces a block entirely on chip:
//   1. left interface rows Z_{d-2}(L) for BL consecutive left indices
//      L = (i_1..i_{d-2}), level by level in LDS (VALU, accumulation
//      precision); for d = 3 these are rows of G_1;
//   2. the middle contraction Z_{d-1}(L, i) = Z_{d-2}(L) G_{d-1}(i) for BI
//      middle indices i, on the matrix cores, into LDS;
//   3. the last contraction out(L, i, :) = Z_{d-1}(L, i) G_d on the matrix
//      cores, stored straight from the accumulators.
// Only the cores are read and only the tensor is written.  Core fragments
// for the matrix cores are fetched two K steps ahead of their use, and each
// feeds every row block of the tile, so global latency overlaps the MFMA
// chains.
// For FP16 the accumulation is FP32 and the interfaces are rounded once to
// FP16 as the inputs of the FP16 products; the FP16 middle and last cores
// are first copied to K-contiguous, zero-padded layouts (KBs to MBs) so a
// lane loads its 8 K values at once.
#include <algorithm>
#include <type_traits>
#include <cstdio>
#include <cstdlib>

#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

struct TTSet {
    const void* core[kMaxD];  // [0] middle core, [1] last core, [2..] left chain
    int64_t ranks[kMaxD + 1];
    int rL, rM, Kp2, Kp3, Rt;
    int ldl, ldf;            // LDS row pitches of Z_{d-2} and Z_{d-1} (elements)
    // staged, zero-padded copies of the middle and last cores, laid out so
    // that a lane's fragment for K step kb sits at a fixed offset plus kb
    // times a uniform stride (see k_stage):
    //   one K value per lane (FP64, FP32): mid [n_mid][Kp2][Rt], last [Kp3][ncp]
    //   eight K values per lane (FP16):     mid [n_mid][Rt][Kp2], last [ncp][Kp3]
    const void* st_mid;
    const void* st_last;
    const void* st_left;     // FP16 wave tiles (d = 3): G_1 rows at pitch Kp2, zero padded
    int zl_off, zf_off;      // byte offsets in LDS
};

struct TTArgs {
    int d;
    int nsets;
    int64_t dims[kMaxD];
    int64_t divs[kMaxD];     // divs[c] = prod of dims[c+1 .. d-3] (left chain)
    int64_t NL, n_mid, n_last;
    int ncp;                 // n_last rounded up to 16 (columns of the staged last core)
    int BL, BI, P, BLpad;
    int chain_rmax, cb_off;  // chain buffers: 2 x BL x chain_rmax (accumulation type)
    int64_t num_L_blocks;
    TTSet set[kTTMaxSets];
    void* out;
    int vec4;
    int vec8;                // FP16 rows of n_last take aligned 16-byte stores (n_last % 8 == 0)
    int lines;               // output rows start on 128-byte lines (n_last * sizeof(T) % 128 == 0)
    int ifast;               // wave tiles: consecutive tiles take consecutive middle indices
};

// Staged copies of the middle core G_{d-1} [rL][n_mid][rM] and the last core
// G_d [rM][n_last], zero padded to Kp2 x Rt and Kp3 x ncp (layouts at TTSet),
// and, when g1 is given, the rows of G_1 [n_1][r_1] at pitch Kp2, zero padded
// (FP16 wave tiles load a lane's eight K values of a row with one aligned
// 16-byte load): one launch for all three.  IDX is the index type: 32-bit
// when every segment is below 2^31 elements (the divisions are much cheaper).
template <typename T, typename IDX>
__global__ __launch_bounds__(256) void k_stage(const T* __restrict__ gmid, const T* __restrict__ glast,
                                               const T* __restrict__ g1, T* __restrict__ smid,
                                               T* __restrict__ slast, T* __restrict__ srows, int64_t n_mid,
                                               int64_t n_last, int64_t n1, int rL, int rM, int r1, int Kp2, int Kp3,
                                               int Rt, int ncp) {
    constexpr bool kcontig = PrecTraits<T>::KPL > 1;
    const int64_t tot_mid = n_mid * Rt * Kp2;
    const int64_t tot_last = (int64_t)ncp * Kp3;
    const int64_t tot_rows = g1 ? n1 * Kp2 : 0;
    const int64_t stride = (int64_t)gridDim.x * 256;
    const int64_t total = tot_mid + tot_last + tot_rows;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total; idx += stride) {
        if (idx < tot_mid) {
            const IDX x = (IDX)idx;
            IDX s, t, i;
            if (kcontig) {
                s = x % (IDX)Kp2;
                t = (x / (IDX)Kp2) % (IDX)Rt;
                i = x / ((IDX)Kp2 * (IDX)Rt);
            } else {
                t = x % (IDX)Rt;
                s = (x / (IDX)Rt) % (IDX)Kp2;
                i = x / ((IDX)Kp2 * (IDX)Rt);
            }
            smid[idx] = ((int)t < rM && (int)s < rL) ? gmid[((int64_t)s * n_mid + (int64_t)i) * rM + (int64_t)t] : T(0);
        } else if (idx < tot_mid + tot_last) {
            const IDX j = (IDX)(idx - tot_mid);
            IDX t, c;
            if (kcontig) {
                t = j % (IDX)Kp3;
                c = j / (IDX)Kp3;
            } else {
                c = j % (IDX)ncp;
                t = j / (IDX)ncp;
            }
            slast[(int64_t)j] = ((int)t < rM && (int64_t)c < n_last) ? glast[(int64_t)t * n_last + (int64_t)c] : T(0);
        } else {
            const IDX j = (IDX)(idx - tot_mid - tot_last);
            const IDX L = j / (IDX)Kp2;
            const int sc = (int)(j - L * (IDX)Kp2);
            srows[(int64_t)j] = sc < r1 ? g1[(int64_t)L * r1 + sc] : T(0);
        }
    }
}

// The same staging for the FP16 wave tiles (K-contiguous layouts, Rt and
// Kp3 at most 96, Kp2 and ncp multiples of 32), transposed through LDS so
// that the global reads run along each core's contiguous index instead of
// gathering along the K index:
//   mid  [n_mid][Rt][Kp2]: workgroup (i, block sb of 32 values of s) reads
//        the rows G_{d-1}(s, i, :) and writes the 16-byte chunks of its 32
//        values of s for every t < Rt;
//   last [ncp][Kp3]: workgroup (block of 32 columns c) reads the rows
//        G_d(t, c0 .. c0 + 31) and writes the chunks of its 32 columns;
//   rows [NL][Kp2]: one chunk of a row of G_1 (or of the left interface)
//        per thread.
// Every thread issues all of its loads before its first LDS write.
constexpr int kStage16T = 96;                 // t extent held in LDS
constexpr int kStage16Ld = kStage16T + 2;     // odd dword pitch: column reads hit distinct banks
constexpr int kStage16Loads = 32 * kStage16T / 256;

__global__ __launch_bounds__(256) void k_stage16(const half_t* __restrict__ gmid, const half_t* __restrict__ glast,
                                                 const half_t* __restrict__ g1, half_t* __restrict__ smid,
                                                 half_t* __restrict__ slast, half_t* __restrict__ srows,
                                                 int64_t n_mid, int64_t n_last, int64_t n1, int rL, int rM, int Kp2,
                                                 int Kp3, int Rt, int ncp, int64_t wg_mid, int64_t wg_last) {
    __shared__ half_t tile[32 * kStage16Ld];
    const int tid = threadIdx.x;
    int64_t wg = blockIdx.x;
    if (wg < wg_mid) {
        const int nsb = Kp2 / 32;
        const int64_t i = wg / nsb;
        const int sb = (int)(wg - i * nsb);
        const int ne = 32 * rM;
        half_t v[kStage16Loads];
#pragma unroll
        for (int q = 0; q < kStage16Loads; ++q) {
            const int e = tid + 256 * q;
            const int r = e / rM, t = e - r * rM, sv = 32 * sb + r;
            v[q] = (e < ne && sv < rL) ? gmid[((int64_t)sv * n_mid + i) * rM + t] : half_t(0);
        }
#pragma unroll
        for (int q = 0; q < kStage16Loads; ++q) {
            const int e = tid + 256 * q;
            const int r = e / rM, t = e - r * rM;
            if (e < ne) tile[r * kStage16Ld + t] = v[q];
        }
        __syncthreads();
        for (int ch = tid; ch < Rt * 4; ch += 256) {
            const int t = ch >> 2, c = ch & 3;
            half8_t w;
#pragma unroll
            for (int j = 0; j < 8; ++j) w[j] = t < rM ? tile[(8 * c + j) * kStage16Ld + t] : half_t(0);
            *reinterpret_cast<half8_t*>(smid + ((i * Rt + t) * (int64_t)Kp2 + 32 * sb + 8 * c)) = w;
        }
        return;
    }
    wg -= wg_mid;
    if (wg < wg_last) {
        const int64_t c0 = wg * 32;
        const int ne = 32 * rM;
        half_t v[kStage16Loads];
#pragma unroll
        for (int q = 0; q < kStage16Loads; ++q) {
            const int e = tid + 256 * q;
            const int t = e >> 5, cc = e & 31;
            v[q] = (e < ne && c0 + cc < n_last) ? glast[(int64_t)t * n_last + c0 + cc] : half_t(0);
        }
#pragma unroll
        for (int q = 0; q < kStage16Loads; ++q) {
            const int e = tid + 256 * q;
            if (e < ne) tile[(e & 31) * kStage16Ld + (e >> 5)] = v[q];
        }
        __syncthreads();
        const int tcs = Kp3 / 8;
        for (int ch = tid; ch < 32 * tcs; ch += 256) {
            const int cc = ch / tcs, tc = ch - cc * tcs;
            half8_t w;
#pragma unroll
            for (int j = 0; j < 8; ++j) w[j] = 8 * tc + j < rM ? tile[cc * kStage16Ld + 8 * tc + j] : half_t(0);
            if (c0 + cc < ncp) *reinterpret_cast<half8_t*>(slast + (c0 + cc) * Kp3 + 8 * tc) = w;
        }
        return;
    }
    wg -= wg_last;
    const int64_t q = wg * 256 + tid;           // chunk of the rows copy
    const int cpr = Kp2 / 8;
    if (q >= n1 * cpr) return;
    const int64_t L = q / cpr;
    const int s0 = 8 * (int)(q - L * cpr);
    half8_t w;
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = s0 + j < rL ? g1[L * rL + s0 + j] : half_t(0);
    *reinterpret_cast<half8_t*>(srows + L * Kp2 + s0) = w;
}

// Side interfaces of a train run by wave tiles as an equivalent three-core
// train (first, middle, last), formed in one launch before the tiles run.
//
// Left interface (mid >= 2):
// Z(p n + i, t) = sum_s z_p(s) G_mid(s, i, t) for every prefix p = (i_1 .. i_{mid-1})
// and n = n_mid, where z_p = G_1(i_1, :) G_2(:, i_2, :) ... is the prefix's
// row vector (sums over s in order in the accumulation precision, as the LDS
// tiles' chain; every entry rounded once to the storage type).  Its rows are
// the left indices (i_1 .. i_mid) in C order, so it takes the place of G_1.
// Left workgroup (q, sp) takes the prefix q = (i_1 .. i_P) of the first P
// digits: it chains the row vector of cores 1 .. P once (a handful of lanes
// per step), then expands cores P+1 .. mid - 1 over all their indices at once
// in LDS (level c holds n_{P+1} ... n_c rows), and writes the rows of the
// last level (core mid) that fall in its share sp of the prefix's rows.
// Taking the serial chain only as deep as the LDS levels require keeps most
// of the work in the wide expansions; the shares keep the grid several
// workgroups per CU.  Every entry is the same sum in the same order whatever
// P is.  The cores are read through the caches (copying the levels' cores
// into LDS first measured slower: 16^6 at ranks 9-25, FP16 9.5 -> 13.1 us).
//
// Right core (two last cores merged, mid = d - 3):
// W(s, i n_d + j) = sum_u G_{d-1}(s, i, u) G_d(u, j), for s < r_{d-2},
// i < n_{d-1}, j < n_d (sum over u in order in the accumulation precision,
// rounded once to the storage type), laid out as a last core of
// r_{d-2} x (n_{d-1} n_d): one thread per entry, in the workgroups after the
// left ones.
struct LeftChain {
    const void* core[kMaxD];
    int64_t dims[kMaxD];
    int64_t ranks[kMaxD + 1];
    int d;                 // cores of the left chain's train: the chain covers cores 1 .. d - 2
    int P;                 // prefix digits per workgroup, 1 <= P <= d - 3
    int shares;            // workgroups per prefix
    int64_t nleft;         // left workgroups (prefixes x shares; 0: no left interface)
    int64_t buf;           // entries of each of the two LDS level buffers
    // right core (rtotal > 0)
    const void* ra;
    const void* rb;
    int64_t rna, rnb, rru, rtotal;
};

template <typename T>
__global__ __launch_bounds__(256) void k_tt_sides(LeftChain lc, T* __restrict__ zo, T* __restrict__ w) {
    using Acc = typename PrecTraits<T>::acc;
    const int tid = threadIdx.x;
    if ((int64_t)blockIdx.x >= lc.nleft) {
        const int64_t e = ((int64_t)blockIdx.x - lc.nleft) * 256 + tid;
        if (e >= lc.rtotal) return;
        const T* ga = static_cast<const T*>(lc.ra);
        const T* gb = static_cast<const T*>(lc.rb);
        const int64_t cols = lc.rna * lc.rnb;
        const int64_t s = e / cols, col = e - s * cols;
        const int64_t i = col / lc.rnb, j = col - i * lc.rnb;
        const T* a = ga + (s * lc.rna + i) * lc.rru;
        Acc sum = 0;
        // 32 loads in flight (from clamped, in-bounds addresses, widened to
        // the accumulation type so no load waits on another), then the
        // products in order
        for (int64_t u0 = 0; u0 < lc.rru; u0 += 16) {
            Acc av[16], bv[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
                const int64_t uc = u0 + u < lc.rru ? u0 + u : lc.rru - 1;
                av[u] = static_cast<Acc>(a[uc]);
                bv[u] = static_cast<Acc>(gb[uc * lc.rnb + j]);
            }
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (u0 + u < lc.rru) sum += av[u] * bv[u];
        }
        w[e] = static_cast<T>(sum);
        return;
    }
    extern __shared__ double4_t lsm[];
    Acc* va = reinterpret_cast<Acc*>(lsm);
    Acc* vb = va + lc.buf;
    const int64_t pfx = (int64_t)blockIdx.x / lc.shares;
    const int sp = (int)((int64_t)blockIdx.x - pfx * lc.shares);
    // the prefix digits i_1 .. i_P, last digit fastest
    int64_t rest = pfx;
    int64_t dig[kMaxD];
    for (int c = lc.P - 1; c >= 0; --c) {
        dig[c] = rest % lc.dims[c];
        rest /= lc.dims[c];
    }
    const T* g0 = static_cast<const T*>(lc.core[0]);
    for (int t = tid; t < lc.ranks[1]; t += 256) va[t] = static_cast<Acc>(g0[dig[0] * lc.ranks[1] + t]);
    __syncthreads();
    for (int c = 1; c < lc.P; ++c) {
        const T* g = static_cast<const T*>(lc.core[c]);
        const int rin = (int)lc.ranks[c], rout = (int)lc.ranks[c + 1];
        const int64_t n = lc.dims[c];
        for (int t = tid; t < rout; t += 256) {
            Acc sum = 0;
#pragma unroll 8
            for (int s2 = 0; s2 < rin; ++s2) sum += va[s2] * static_cast<Acc>(g[((int64_t)s2 * n + dig[c]) * rout + t]);
            vb[t] = sum;
        }
        __syncthreads();
        Acc* tmp = va;
        va = vb;
        vb = tmp;
    }
    // expansions: level c holds rows (i_{P+1} .. i_{c+1}) x r_{c+1}
    int64_t rows = 1;
    for (int c = lc.P; c < lc.d - 3; ++c) {
        const int rin = (int)lc.ranks[c], rout = (int)lc.ranks[c + 1];
        const int n = (int)lc.dims[c];
        const int total = (int)(rows * n * rout);   // entries of the level: fits LDS
        const T* g = static_cast<const T*>(lc.core[c]);
        for (int e = tid; e < total; e += 256) {
            const int ri = e / rout, t = e - ri * rout;
            const int row = ri / n, i = ri - row * n;
            const Acc* z = va + row * rin;
            Acc sum = 0;
#pragma unroll 8
            for (int s2 = 0; s2 < rin; ++s2) sum += z[s2] * static_cast<Acc>(g[((int64_t)s2 * n + i) * rout + t]);
            vb[e] = sum;
        }
        __syncthreads();
        Acc* tmp = va;
        va = vb;
        vb = tmp;
        rows *= n;
    }
    // last level (core mid): this workgroup's share of the prefix's rows
    const int c = lc.d - 3;
    const int rin = (int)lc.ranks[c], rout = (int)lc.ranks[c + 1];
    const int64_t n = lc.dims[c];
    const int64_t fin = rows * n;                               // rows of the prefix
    const int64_t per = (fin + lc.shares - 1) / lc.shares;
    const int64_t r0 = (int64_t)sp * per;
    const int64_t r1 = (r0 + per < fin) ? r0 + per : fin;
    T* dst = zo + pfx * fin * rout;
    const T* g = static_cast<const T*>(lc.core[c]);
    for (int64_t e = r0 * rout + tid; e < r1 * rout; e += 256) {
        const int64_t ri = e / rout;
        const int t = (int)(e - ri * rout);
        const int64_t row = ri / n, i = ri - row * n;
        const Acc* z = va + row * rin;
        Acc sum = 0;
#pragma unroll 8
        for (int s2 = 0; s2 < rin; ++s2) sum += z[s2] * static_cast<Acc>(g[((int64_t)s2 * n + i) * rout + t]);
        dst[e] = static_cast<T>(sum);
    }
}

// Prefix depth and shares of the left interface: the smallest P whose
// expansion levels fit both LDS buffers (32 KB) and cost a workgroup no more
// multiply-adds than its share of the last level (each share repeats them);
// P = d - 3 (no expansion level) is always possible.  The shares bring the
// grid to about 1024 workgroups, with at least 16 rows each.
static void left_split(LeftChain& lc, size_t acc_bytes) {
    constexpr size_t kLdsBudget = (size_t)32 << 10;
    constexpr int64_t kTargetWgs = 1024, kMinShareRows = 16;
    const int d = lc.d;
    const int64_t* dims = lc.dims;
    const int64_t* ranks = lc.ranks;
    for (int P = 1; P <= d - 3; ++P) {
        int64_t npfx = 1, buf = 1, rows = 1, inter = 0;
        for (int c = 0; c < P; ++c) npfx *= dims[c];
        for (int c = 1; c <= P; ++c) buf = std::max(buf, ranks[c]);
        for (int c = P; c < d - 3; ++c) {
            rows *= dims[c];
            buf = std::max(buf, rows * ranks[c + 1]);
            inter += rows * ranks[c + 1] * ranks[c];
        }
        const int64_t fin = rows * dims[d - 3];
        int64_t shares = (kTargetWgs + npfx - 1) / npfx;
        shares = std::min(shares, std::max<int64_t>(1, fin / kMinShareRows));
        shares = std::min<int64_t>(shares, 65535);
        const int64_t last = (fin + shares - 1) / shares * ranks[d - 2] * ranks[d - 3];
        if (P < d - 3 && (2 * (size_t)buf * acc_bytes > kLdsBudget || inter > last)) continue;
        lc.P = P;
        lc.shares = (int)shares;
        lc.nleft = npfx * shares;
        lc.buf = buf;
        break;
    }
}

// Fragment address of the staged middle core for middle index i (clamped
// into range: rows past the tensor are discarded at the store), output
// column t, this lane's K group g; step kb adds kb * mid_step<T>(S).
template <typename T>
__device__ __forceinline__ const T* mid_base(const TTSet& S, int64_t n_mid, int64_t i, int t, int g) {
    const T* st = static_cast<const T*>(S.st_mid);
    const int64_t ic = i < n_mid ? i : n_mid - 1;
    if constexpr (PrecTraits<T>::KPL > 1) return st + (ic * S.Rt + t) * S.Kp2 + g * PrecTraits<T>::KPL;
    else return st + (ic * S.Kp2 + g) * S.Rt + t;
}
template <typename T>
__device__ __forceinline__ int64_t mid_step(const TTSet& S) {
    return PrecTraits<T>::KPL > 1 ? (int64_t)PrecTraits<T>::KB : (int64_t)PrecTraits<T>::KB * S.Rt;
}
// Same for the staged last core, output column c (< ncp).
template <typename T>
__device__ __forceinline__ const T* last_base(const TTSet& S, int ncp, int64_t c, int g) {
    const T* st = static_cast<const T*>(S.st_last);
    if constexpr (PrecTraits<T>::KPL > 1) return st + c * S.Kp3 + g * PrecTraits<T>::KPL;
    else return st + (int64_t)g * ncp + c;
}
template <typename T>
__device__ __forceinline__ int64_t last_step(int ncp) {
    return PrecTraits<T>::KPL > 1 ? (int64_t)PrecTraits<T>::KB : (int64_t)PrecTraits<T>::KB * ncp;
}
template <typename T>
__device__ __forceinline__ typename PrecTraits<T>::frag core_frag(const T* p) {
    if constexpr (PrecTraits<T>::KPL > 1) return *reinterpret_cast<const typename PrecTraits<T>::frag*>(p);
    else return *p;
}

// Left interface rows Z_{d-2}(L) for L in [L0, L0 + BL) into Zl[BLpad][Kp2]
// (storage type; rows >= BL and columns >= rL are zero).  lcore[c] is core c
// of the left chain.
template <typename T, int NT>
__device__ void build_left(const TTArgs& a, const TTSet& S, const void* const* lcore, int64_t L0, T* Zl,
                           typename PrecTraits<T>::acc* cb0, typename PrecTraits<T>::acc* cb1) {
    using Acc = typename PrecTraits<T>::acc;
    const int tid = threadIdx.x;
    const int total = a.BLpad * S.Kp2;   // rows of Zl have pitch S.ldl
    if (a.d == 2) {
        for (int idx = tid; idx < total; idx += NT) {
            const int Lr = idx / S.Kp2, s = idx % S.Kp2;
            Zl[Lr * S.ldl + s] = (idx == 0) ? T(1) : T(0);
        }
        return;
    }
    if (a.d == 3) {
        const T* g1 = static_cast<const T*>(lcore[0]);
        for (int idx = tid; idx < total; idx += NT) {
            const int Lr = idx / S.Kp2, s = idx % S.Kp2;
            const int64_t L = L0 + Lr;
            Zl[Lr * S.ldl + s] = (Lr < a.BL && L < a.NL && s < S.rL) ? g1[L * S.rL + s] : T(0);
        }
        return;
    }
    const int64_t Lend = (L0 + a.BL < a.NL) ? L0 + a.BL : a.NL;
    Acc* cur = cb0;
    Acc* nxt = cb1;
    int64_t qlo_prev = 0;
    for (int c = 0; c <= a.d - 3; ++c) {
        const int64_t D = a.divs[c];
        const int64_t qlo = L0 / D, qhi = (Lend - 1) / D;
        const int cnt = (int)(qhi - qlo + 1);
        const int r1 = (int)S.ranks[c + 1];
        const int64_t nc = a.dims[c];
        const T* g = static_cast<const T*>(lcore[c]);
        if (c == 0) {
            for (int idx = tid; idx < cnt * r1; idx += NT) {
                const int ql = idx / r1, t = idx % r1;
                nxt[ql * a.chain_rmax + t] = to_acc(g[(qlo + ql) * r1 + t]);
            }
        } else {
            const int r0 = (int)S.ranks[c];
            for (int idx = tid; idx < cnt * r1; idx += NT) {
                const int ql = idx / r1, t = idx % r1;
                const int64_t q = qlo + ql;
                const int pl = (int)(q / nc - qlo_prev);
                const int64_t i = q % nc;
                const Acc* zrow = cur + pl * a.chain_rmax;
                Acc sum = 0;
                for (int s = 0; s < r0; ++s) sum += zrow[s] * to_acc(g[((int64_t)s * nc + i) * r1 + t]);
                nxt[ql * a.chain_rmax + t] = sum;
            }
        }
        __syncthreads();
        Acc* tmp = cur;
        cur = nxt;
        nxt = tmp;
        qlo_prev = qlo;
    }
    for (int idx = tid; idx < total; idx += NT) {
        const int Lr = idx / S.Kp2, s = idx % S.Kp2;
        const bool ok = (Lr < a.BL) && (L0 + Lr < a.NL) && (s < S.rL);
        Zl[Lr * S.ldl + s] = ok ? to_storage<T>(cur[Lr * a.chain_rmax + s]) : T(0);
    }
    __syncthreads();   // the chain buffers are reused by the next set
}

// acc[c][j] += sum_kb A_c(kb) B_j(kb) for c < NC, j < NJ, over nkb >= 1 K
// steps (with SWAP the products are B_j A_c: the accumulators then hold the
// transposed blocks).  Four register sets hold the A fragments (core
// fragments from global memory) of steps kb .. kb+3 and two sets the B
// fragments (LDS) of steps kb, kb+1; each set is refilled right after the
// step that used it, for the step four (A) or two (B) later, so no register
// is copied and every load has several steps of matrix-core work to arrive.
// Indices past the end are clamped, so the load sequence has no branches.
template <typename T, int NC, int NJ, bool SWAP = false, class AF, class BF>
__device__ __forceinline__ void mma_chain(AF afrag, BF bfrag, int nkb,
                                          typename PrecTraits<T>::accv (&acc)[NC][NJ]) {
    using Frag = typename PrecTraits<T>::frag;
    auto cl = [nkb](int k) { return k < nkb ? k : nkb - 1; };
    Frag x0[NC], x1[NC], y0[NC], y1[NC], be[NJ], bo[NJ];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        x0[c] = afrag(c, 0);
        x1[c] = afrag(c, cl(1));
        y0[c] = afrag(c, cl(2));
        y1[c] = afrag(c, cl(3));
    }
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
        be[j] = bfrag(j, 0);
        bo[j] = bfrag(j, cl(1));
    }
    auto step = [&](Frag (&a)[NC], Frag (&b)[NJ]) {
#pragma unroll
        for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int j = 0; j < NJ; ++j) acc[c][j] = SWAP ? mfma(b[j], a[c], acc[c][j]) : mfma(a[c], b[j], acc[c][j]);
    };
    auto refill_a = [&](Frag (&a)[NC], int k) {
#pragma unroll
        for (int c = 0; c < NC; ++c) a[c] = afrag(c, cl(k));
    };
    auto refill_b = [&](Frag (&b)[NJ], int k) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) b[j] = bfrag(j, cl(k));
    };
    // the scheduling barriers keep each refill right behind its step (the
    // scheduler would otherwise bunch the loads late and shorten their lead)
    int kb = 0;
    for (; kb + 3 < nkb; kb += 4) {
        step(x0, be);
        refill_a(x0, kb + 4);
        refill_b(be, kb + 2);
        __builtin_amdgcn_sched_barrier(0);
        step(x1, bo);
        refill_a(x1, kb + 5);
        refill_b(bo, kb + 3);
        __builtin_amdgcn_sched_barrier(0);
        step(y0, be);
        refill_a(y0, kb + 6);
        refill_b(be, kb + 4);
        __builtin_amdgcn_sched_barrier(0);
        step(y1, bo);
        refill_a(y1, kb + 7);
        refill_b(bo, kb + 5);
        __builtin_amdgcn_sched_barrier(0);
    }
    // remaining 1 to 3 steps: x0, x1, y0 hold A of steps kb .. kb+2
    if (kb < nkb) {
        step(x0, be);
        if (kb + 1 < nkb) {
            refill_b(be, kb + 2);
            step(x1, bo);
            if (kb + 2 < nkb) step(y0, be);
        }
    }
}

// Middle product of one tile, Z_{d-1}(L, i) = Z_{d-2}(L) G_{d-1}(i), from Zl
// into Zf (rounded to T): work units (il, tb) over the four waves, each
// feeding NLB accumulators.  Zf columns at and beyond min(Rt, Kp3) are never
// written (the caller clears them once).
template <typename T, int NLB>
__device__ __forceinline__ void middle_product(const TTArgs& a, const TTSet& S, const T* Zl, T* Zf, int64_t i0,
                                               int wave, int r, int g) {
    using AccV = typename PrecTraits<T>::accv;
    constexpr int KB = PrecTraits<T>::KB, KPL = PrecTraits<T>::KPL;
    const int n_tb = S.Rt / 16;
    const int tcap = (S.Rt < S.Kp3) ? S.Rt : S.Kp3;
    for (int u = wave; u < a.BI * n_tb; u += 4) {
        const int il = u / n_tb, tb = u % n_tb;
        const int64_t i = i0 + il;
        AccV acc[1][NLB];
#pragma unroll
        for (int j = 0; j < NLB; ++j) acc[0][j] = zero_accv<AccV>();
        const T* mb = mid_base<T>(S, a.n_mid, i, tb * 16 + r, g);
        const int64_t ms = mid_step<T>(S);
        mma_chain<T, 1, NLB>(
            [&](int, int kb) { return core_frag<T>(mb + kb * ms); },
            [&](int j, int kb) { return load_frag<T>(Zl + (j * 16 + r) * S.ldl + kb * KB + g * KPL); },
            S.Kp2 / KB, acc);
#pragma unroll
        for (int j = 0; j < NLB; ++j) {
            const int Lr = j * 16 + r;
            if (Lr >= a.BL) continue;
            T* dst = Zf + (Lr * a.BI + il) * S.ldf;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int t = tb * 16 + acc_row<T>(g, v);
                if (t < tcap) dst[t] = to_storage<T>(acc[0][j][v]);
            }
        }
    }
}

// Last product of column blocks NCB*cp .. NCB*cp + NCB - 1 against Zf; with
// SWAP the accumulators hold the transposed blocks (tensor rows in the
// accumulator rows).
template <typename T, int NCB, int NPB, bool SWAP>
__device__ __forceinline__ void last_product(const TTArgs& a, const TTSet& S, const T* Zf, int cp, int r, int g,
                                             typename PrecTraits<T>::accv (&acc)[NCB][NPB]) {
    constexpr int KB = PrecTraits<T>::KB, KPL = PrecTraits<T>::KPL;
#pragma unroll
    for (int c = 0; c < NCB; ++c)
#pragma unroll
        for (int j = 0; j < NPB; ++j) acc[c][j] = zero_accv<typename PrecTraits<T>::accv>();
    const T* lb0 = last_base<T>(S, a.ncp, (int64_t)(NCB * cp) * 16 + r, g);
    const int64_t lstep = last_step<T>(a.ncp);
    const int64_t cstep = (KPL > 1) ? (int64_t)16 * S.Kp3 : 16;   // next column block
    mma_chain<T, NCB, NPB, SWAP>(
        [&](int c, int kb) { return core_frag<T>(lb0 + c * cstep + kb * lstep); },
        [&](int j, int kb) { return load_frag<T>(Zf + (j * 16 + r) * S.ldf + kb * KB + g * KPL); },
        S.Kp3 / KB, acc);
}

// NPB = P / 16 row blocks of the tile, NLB = BLpad / 16 row blocks of the
// left interface (both fixed at compile time, so that the matrix-core loops
// carry no per-product branches).
template <typename T, int NPB, int NLB>
__global__ __launch_bounds__(256) void k_tt_fused(TTArgs a) {
    using AccV = typename PrecTraits<T>::accv;
    using Acc = typename PrecTraits<T>::acc;
    constexpr int KPL = PrecTraits<T>::KPL;
    extern __shared__ double4_t smem_v[];
    char* smem = reinterpret_cast<char*>(smem_v);
    const TTSet& S = a.set[0];
    T* Zl = reinterpret_cast<T*>(smem + S.zl_off);
    T* Zf = reinterpret_cast<T*>(smem + S.zf_off);
    Acc* cb0 = reinterpret_cast<Acc*>(smem + a.cb_off);
    Acc* cb1 = cb0 + (size_t)a.BL * a.chain_rmax;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, g = lane >> 4;
    const int64_t i0 = (int64_t)blockIdx.x * a.BI;
    const int n_cb = (int)((a.n_last + 15) / 16);

    for (int idx = tid; idx < a.P * S.ldf; idx += 256) Zf[idx] = T(0);

    // last product: NCB 16-column blocks per wave at a time (two for the
    // FP64 / FP32 matrix-core chains, one for FP16, whose short K keeps the
    // work per block small); each core fragment feeds the NPB row blocks.
    // FP64 accumulators hold rows g + 4v of a block: computing the
    // transposed block makes each lane's values one tensor column of four
    // rows, and lanes 0..15 sixteen consecutive columns.
    constexpr int NCB = (KPL == 8) ? 1 : 2;
    constexpr bool kRowsOut = !AccRowsContiguous<T>::value;

    for (int64_t lb = blockIdx.y; lb < a.num_L_blocks; lb += gridDim.y) {
        const int64_t L0 = lb * a.BL;
        __syncthreads();   // readers of the previous block are done
        build_left<T, 256>(a, S, S.core + 2, L0, Zl, cb0, cb1);
        __syncthreads();
        middle_product<T, NLB>(a, S, Zl, Zf, i0, wave, r, g);
        __syncthreads();

        for (int cp = wave; cp < (n_cb + NCB - 1) / NCB; cp += 4) {
            AccV acc[NCB][NPB];
            last_product<T, NCB, NPB, kRowsOut>(a, S, Zf, cp, r, g, acc);
            if constexpr (kRowsOut) {
                // lane holds tensor rows p = pb*16 + acc_row(g, v) of column
                // NCB*cp*16 + 16c + r: each store instruction writes whole
                // 128-byte row segments
#pragma unroll
                for (int c = 0; c < NCB; ++c) {
                    const int64_t col = (int64_t)(NCB * cp + c) * 16 + r;
                    if (col >= a.n_last) continue;
#pragma unroll
                    for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const int p = pb * 16 + acc_row<T>(g, v);
                            const int Lr = (a.BI == 1) ? p : p / a.BI, il = (a.BI == 1) ? 0 : p % a.BI;
                            const int64_t L = L0 + Lr, i = i0 + il;
                            if (Lr >= a.BL || L >= a.NL || i >= a.n_mid) continue;
                            static_cast<T*>(a.out)[(L * a.n_mid + i) * a.n_last + col] = to_storage<T>(acc[c][pb][v]);
                        }
                }
            } else {
#pragma unroll
                for (int c = 0; c < NCB; ++c) {
                    const int64_t cbase = (int64_t)(NCB * cp + c) * 16;
                    if (cbase >= a.n_last) continue;
#pragma unroll
                    for (int pb = 0; pb < NPB; ++pb) {
                        const int p = pb * 16 + r;
                        const int Lr = p / a.BI, il = p % a.BI;
                        const int64_t L = L0 + Lr, i = i0 + il;
                        if (Lr >= a.BL || L >= a.NL || i >= a.n_mid) continue;
                        T* dst = static_cast<T*>(a.out) + (L * a.n_mid + i) * a.n_last + cbase;
                        if (a.vec4 && cbase + 4 * g + 3 < a.n_last) {
                            typedef T vec_t __attribute__((ext_vector_type(4)));
                            vec_t w;
#pragma unroll
                            for (int v = 0; v < 4; ++v) w[v] = to_storage<T>(acc[c][pb][v]);
                            *reinterpret_cast<vec_t*>(dst + 4 * g) = w;
                        } else {
#pragma unroll
                            for (int v = 0; v < 4; ++v) {
                                const int row = acc_row<T>(g, v);
                                if (cbase + row < a.n_last) dst[row] = to_storage<T>(acc[c][pb][v]);
                            }
                        }
                    }
                }
            }
        }
    }
}

// Left interface rows of a tile for d = 3 (rows of G_1), fetched into
// registers ahead of their use.  The BLpad = 16 NLB rows are spread over
// the 256 threads, TPR = 256 / BLpad threads per row; entry e of a thread is
// column tid % TPR + TPR e of row tid / TPR (e < NE covers Kp2 <= TPR NE).
// The loads are unconditional (clamped addresses) and masked only when
// stored, so that they stay in flight across the work that runs meanwhile.
template <int NLB, int NE>
__device__ __forceinline__ void fetch_left3(const TTArgs& a, const TTSet& S, int64_t L0, int tid, double (&v)[NE]) {
    constexpr int TPR = 256 / (16 * NLB);
    const double* g1 = static_cast<const double*>(S.core[2]);
    const int Lr = tid / TPR, c0 = tid % TPR;
    const int64_t L = L0 + Lr;
    const double* row = g1 + ((Lr < a.BL && L < a.NL) ? L : 0) * S.rL;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        if (TPR * e >= S.Kp2) break;
        const int c = c0 + TPR * e;
        v[e] = row[c < S.rL ? c : 0];
    }
}
template <int NLB, int NE>
__device__ __forceinline__ void store_left3(const TTArgs& a, const TTSet& S, int64_t L0, int tid,
                                            const double (&v)[NE], double* Zl) {
    constexpr int TPR = 256 / (16 * NLB);
    const int Lr = tid / TPR, c0 = tid % TPR;
    const bool rok = Lr < a.BL && L0 + Lr < a.NL;
    double* dst = Zl + Lr * S.ldl + c0;
#pragma unroll
    for (int e = 0; e < NE; ++e) {
        if (TPR * e >= S.Kp2) break;
        const int c = c0 + TPR * e;
        if (c < S.Kp2) dst[TPR * e] = (rok && c < S.rL) ? v[e] : 0.0;
    }
}

// acc[q][j] += sum_kb B_q(kb, j) A_q(kb) for the NS core sets at once
// (transposed blocks, FP64): one chain whose steps issue the products of
// every set, with the register rings of mma_chain (four A sets from global
// memory, two B sets from LDS, each refilled right behind its step).
template <int NS, int NJ, class AF, class BF>
__device__ __forceinline__ void mma_chain_sets(AF afrag, BF bfrag, int nkb, double4_t (&acc)[NS][NJ]) {
    auto cl = [nkb](int k) { return k < nkb ? k : nkb - 1; };
    double x0[NS], x1[NS], y0[NS], y1[NS], be[NS][NJ], bo[NS][NJ];
#pragma unroll
    for (int q = 0; q < NS; ++q) {
        x0[q] = afrag(q, 0);
        x1[q] = afrag(q, cl(1));
        y0[q] = afrag(q, cl(2));
        y1[q] = afrag(q, cl(3));
    }
#pragma unroll
    for (int q = 0; q < NS; ++q)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            be[q][j] = bfrag(q, j, 0);
            bo[q][j] = bfrag(q, j, cl(1));
        }
    auto step = [&](double (&x)[NS], double (&b)[NS][NJ]) {
#pragma unroll
        for (int q = 0; q < NS; ++q)
#pragma unroll
            for (int j = 0; j < NJ; ++j) acc[q][j] = mfma(b[q][j], x[q], acc[q][j]);
    };
    auto refill_a = [&](double (&x)[NS], int k) {
#pragma unroll
        for (int q = 0; q < NS; ++q) x[q] = afrag(q, cl(k));
    };
    auto refill_b = [&](double (&b)[NS][NJ], int k) {
#pragma unroll
        for (int q = 0; q < NS; ++q)
#pragma unroll
            for (int j = 0; j < NJ; ++j) b[q][j] = bfrag(q, j, cl(k));
    };
    int kb = 0;
    for (; kb + 3 < nkb; kb += 4) {
        step(x0, be);
        refill_a(x0, kb + 4);
        refill_b(be, kb + 2);
        __builtin_amdgcn_sched_barrier(0);
        step(x1, bo);
        refill_a(x1, kb + 5);
        refill_b(bo, kb + 3);
        __builtin_amdgcn_sched_barrier(0);
        step(y0, be);
        refill_a(y0, kb + 6);
        refill_b(be, kb + 4);
        __builtin_amdgcn_sched_barrier(0);
        step(y1, bo);
        refill_a(y1, kb + 7);
        refill_b(bo, kb + 5);
        __builtin_amdgcn_sched_barrier(0);
    }
    if (kb < nkb) {
        step(x0, be);
        if (kb + 1 < nkb) {
            refill_b(be, kb + 2);
            step(x1, bo);
            if (kb + 2 < nkb) step(y0, be);
        }
    }
}

// TT certificate (Thm. thm:tt_conditional) without dense reconstructions:
// for each tile the FP64 reconstructions from the base cores (set 0), the
// augmented cores (set 1) and the widened rounded augmented cores (set 2)
// are formed on chip and compared with T.  The three middle products run
// one after the other through the shared Z_{d-2} buffer (for d = 3 the next
// set's rows of G_1 are fetched while the current product runs); the last
// products of the three sets share one matrix-core chain per column block,
// with the block's values of T fetched before the chain.  All sets use one
// K extent for the last product (the largest; the staged cores and the Z_{d-1}
// columns beyond a set's rank are zero).  Workgroup w writes
// part[s * nparts + w] for the five sums
//   s = 0 ||T - T_R||^2, 1 ||T - T_R+||^2, 2 ||T_R+ - T^_R+||^2,
//       3 ||T - T^_R+||^2, 4 ||T||^2,
// each accumulated per lane in a fixed order and combined in wave order.
template <int NPB, int NLB>
__global__ __launch_bounds__(256) void k_tt_cert(TTArgs a, const double* __restrict__ Tref,
                                                 double* __restrict__ part, int64_t nparts) {
    using T = double;
    using AccV = double4_t;
    constexpr int NE = 16;   // prefetched G_1 entries per thread (d = 3)
    extern __shared__ double4_t smem_v[];
    char* smem = reinterpret_cast<char*>(smem_v);
    T* Zl = reinterpret_cast<T*>(smem);
    double* cb0 = reinterpret_cast<double*>(smem + a.cb_off);
    double* cb1 = cb0 + (size_t)a.BL * a.chain_rmax;
    __shared__ double red[4][5];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t i0 = (int64_t)blockIdx.x * a.BI;
    const int n_cb = (int)((a.n_last + 15) / 16);
    const T* Zf0 = reinterpret_cast<const T*>(smem + a.set[0].zf_off);
    const T* Zf1 = reinterpret_cast<const T*>(smem + a.set[1].zf_off);
    const T* Zf2 = reinterpret_cast<const T*>(smem + a.set[2].zf_off);
    // d = 3 with every set's rows within the prefetch registers
    bool pre = a.d == 3 && a.BLpad == 16 * NLB;
    for (int q = 0; q < 3; ++q) pre = pre && a.set[q].Kp2 <= (256 / (16 * NLB)) * NE;

    for (int q = 0; q < 3; ++q) {
        T* Zf = reinterpret_cast<T*>(smem + a.set[q].zf_off);
        for (int idx = tid; idx < a.P * a.set[q].ldf; idx += 256) Zf[idx] = T(0);
    }
    double sum[5] = {0.0, 0.0, 0.0, 0.0, 0.0};
    const int Kp3 = a.set[0].Kp3;   // common to the three sets
    const int nkb = Kp3 / 4;

    for (int64_t lb = blockIdx.y; lb < a.num_L_blocks; lb += gridDim.y) {
        const int64_t L0 = lb * a.BL;
        // per-block copies of the thread index: addresses derived from them
        // are formed in the phase that uses them instead of being kept live
        // across the whole loop
        int tm = tid;
        asm volatile("" : "+v"(tm));
        const int rm = tm & 15, gm = (tm & 63) >> 4;
        double v[NE];
        if (pre) fetch_left3<NLB, NE>(a, a.set[0], L0, tm, v);
        for (int q = 0; q < 3; ++q) {
            const TTSet& S = a.set[q];
            __syncthreads();   // Zl (and, for q = 0, every Zf) is free again
            if (pre) {
                store_left3<NLB, NE>(a, S, L0, tm, v, Zl);
                __syncthreads();
                if (q < 2) fetch_left3<NLB, NE>(a, a.set[q + 1], L0, tm, v);
            } else {
                build_left<T, 256>(a, S, S.core + 2, L0, Zl, cb0, cb1);
                __syncthreads();
            }
            middle_product<T, NLB>(a, S, Zl, reinterpret_cast<T*>(smem + S.zf_off), i0, wave, rm, gm);
        }
        __syncthreads();

        int tl = tid;
        asm volatile("" : "+v"(tl));
        const int r = tl & 15, g = (tl & 63) >> 4;
        for (int cp = wave; cp < n_cb; cp += 4) {
            // transposed blocks: lane holds rows p = pb*16 + g + 4v of column col
            const int64_t col = (int64_t)cp * 16 + r;
            double tv[NPB][4];
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
                for (int v4 = 0; v4 < 4; ++v4) {
                    const int p = pb * 16 + acc_row<T>(g, v4);
                    const int Lr = (a.BI == 1) ? p : p / a.BI, il = (a.BI == 1) ? 0 : p % a.BI;
                    const int64_t L = L0 + Lr, i = i0 + il;
                    const bool ok = col < a.n_last && Lr < a.BL && L < a.NL && i < a.n_mid;
                    tv[pb][v4] = Tref[ok ? (L * a.n_mid + i) * a.n_last + col : 0];
                }
            AccV acc[3][NPB];
#pragma unroll
            for (int q = 0; q < 3; ++q)
#pragma unroll
                for (int j = 0; j < NPB; ++j) acc[q][j] = zero_accv<AccV>();
            const T* lb0 = last_base<T>(a.set[0], a.ncp, col, g);
            const T* lb1 = last_base<T>(a.set[1], a.ncp, col, g);
            const T* lb2 = last_base<T>(a.set[2], a.ncp, col, g);
            const int64_t lstep = last_step<T>(a.ncp);
            mma_chain_sets<3, NPB>(
                [&](int q, int kb) { return (q == 0 ? lb0 : (q == 1 ? lb1 : lb2))[kb * lstep]; },
                [&](int q, int j, int kb) {
                    const T* Zf = q == 0 ? Zf0 : (q == 1 ? Zf1 : Zf2);
                    return Zf[(j * 16 + r) * a.set[q].ldf + kb * 4 + g];
                },
                nkb, acc);
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
                for (int v4 = 0; v4 < 4; ++v4) {
                    const int p = pb * 16 + acc_row<T>(g, v4);
                    const int Lr = (a.BI == 1) ? p : p / a.BI, il = (a.BI == 1) ? 0 : p % a.BI;
                    const int64_t L = L0 + Lr, i = i0 + il;
                    const bool ok = col < a.n_last && Lr < a.BL && L < a.NL && i < a.n_mid;
                    // rows outside the tensor compare zero with zero
                    const double t = ok ? tv[pb][v4] : 0.0;
                    const double r0 = ok ? acc[0][pb][v4] : 0.0;
                    const double r1 = ok ? acc[1][pb][v4] : 0.0;
                    const double r2 = ok ? acc[2][pb][v4] : 0.0;
                    const double d0 = t - r0, d1 = t - r1, d2 = r1 - r2, d3 = t - r2;
                    sum[0] += d0 * d0;
                    sum[1] += d1 * d1;
                    sum[2] += d2 * d2;
                    sum[3] += d3 * d3;
                    sum[4] += t * t;
                }
        }
        __syncthreads();   // the Zf buffers are rewritten for the next block
    }

#pragma unroll
    for (int s = 0; s < 5; ++s) {
        const double w = wave_sum(sum[s]);
        if (lane == 0) red[wave][s] = w;
    }
    __syncthreads();
    if (tid < 5) {
        const int64_t wg = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
        part[tid * nparts + wg] = ((red[0][tid] + red[1][tid]) + red[2][tid]) + red[3][tid];
    }
}

// ---------------------------------------------------------------------------
// Wave-tile TT certificate for d = 3 whose last-product K extent fits the
// registers (Kp3 = 4 NKB <= 68).  Each wave owns 16 rows L0 .. L0+15 of G_1
// for one middle index i and all n_3 columns, and works alone: no LDS and no
// barriers.  For each set it forms Z_2(L, i, :) = G_1(L, :) G_2(:, i, :) as
// the transposed product G_2(:, i, :)^T G_1(L, :)^T on the matrix cores: the
// accumulator of column block tb holds, in lane (r, g), value v,
// Z_2(L0 + r, i, 16 tb + g + 4 v), which is exactly the A fragment of the
// last product for K step kb = 4 tb + v (lane (r, g) supplies
// Z_2(L0 + r, i, 4 kb + g)).  So the three Z_2 tiles stay in registers, and
// the last products of the three sets run as one fully unrolled chain per
// 16-column block of the output; the staged last-core fragments are fetched
// four steps ahead, the last four steps of a block fetching the first four
// of the next.

// Load at a uniform base plus a per-lane byte offset (one 32-bit register
// per lane; the step offsets stay in scalar registers).
template <typename T>
__device__ __forceinline__ T ld_off(const T* base, uint32_t byte_off) {
    return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + byte_off);
}

// The middle products of all NPB row blocks of a tile (FP64 or FP32) in one
// chain: acc[pb][tb] for the NT column blocks of Z_2 over ceil(r_1 / 4) K
// steps; each step multiplies the step's G_2 fragments (fetched once, for
// every row block; lane (r, g) of step kb reads G_2(4 kb + g, i, 16 tb + r):
// sixteen consecutive entries per lane group) with each row block's G_1
// fragment.  Indices past the ranks are clamped into the cores, so the loads
// are unconditional.  K values past r_1 occur in the last step only, whose
// G_1 values there are replaced by zero; Z_2 columns past r_2 (formed from
// clamped copies of the last column) are set to zero once the chain ends.
template <typename T, int NT, int NPB>
__device__ __forceinline__ void middle_w_tile(const TTArgs& a, const TTSet& S, int64_t i, int64_t L0, int r, int g,
                                              typename PrecTraits<T>::accv (&acc)[NPB][NT]) {
    using AccV = typename PrecTraits<T>::accv;
    const T* g2 = static_cast<const T*>(S.core[0]) + i * S.rM;   // uniform
    const uint32_t ld2 = (uint32_t)(a.n_mid * S.rM);
    const T* zr[NPB];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
        const int64_t row = (L0 + 16 * pb + r < a.NL) ? L0 + 16 * pb + r : a.NL - 1;
        zr[pb] = static_cast<const T*>(S.core[2]) + row * S.rL;
    }
    const int klast = S.rL - 1, tlast = S.rM - 1;
    const int nkb = (S.rL + 3) / 4;
    uint32_t tcol[NT];
#pragma unroll
    for (int tb = 0; tb < NT; ++tb) {
        const int t = 16 * tb + r;
        tcol[tb] = (uint32_t)(t < tlast ? t : tlast);
    }
    auto cl = [nkb](int k) { return k < nkb ? k : nkb - 1; };
    auto fetch = [&](T (&x)[NT], T (&b)[NPB], int kb) {
        const int sk = 4 * cl(kb) + g;
        const int sc = sk < klast ? sk : klast;
        const uint32_t ro = (uint32_t)sc * ld2;
#pragma unroll
        for (int tb = 0; tb < NT; ++tb) x[tb] = ld_off(g2, (ro + tcol[tb]) * (uint32_t)sizeof(T));
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) b[pb] = zr[pb][sc];
    };
    // MASK: a step that may hold K values past r_1 (the tail of the chain)
    auto step = [&](const T (&x)[NT], const T (&b)[NPB], int kb, auto mask) {
        T bm[NPB];
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) {
            if constexpr (decltype(mask)::value) bm[pb] = 4 * kb + g <= klast ? b[pb] : T(0);
            else bm[pb] = b[pb];
        }
#pragma unroll
        for (int tb = 0; tb < NT; ++tb)
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb) acc[pb][tb] = mfma(x[tb], bm[pb], acc[pb][tb]);
    };
    constexpr std::false_type kFull{};
    constexpr std::true_type kTail{};
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
        for (int tb = 0; tb < NT; ++tb) acc[pb][tb] = zero_accv<AccV>();
    T x0[NT], x1[NT], y0[NT], y1[NT], b0[NPB], b1[NPB], c0[NPB], c1[NPB];
    // steps past the end are neither fetched nor computed (uniform branches)
    fetch(x0, b0, 0);
    if (nkb > 1) fetch(x1, b1, 1);
    if (nkb > 2) fetch(y0, c0, 2);
    if (nkb > 3) fetch(y1, c1, 3);
    int kb = 0;
    for (; kb + 7 < nkb; kb += 4) {   // every refill lies inside the chain
        step(x0, b0, kb, kFull);
        fetch(x0, b0, kb + 4);
        __builtin_amdgcn_sched_barrier(0);
        step(x1, b1, kb + 1, kFull);
        fetch(x1, b1, kb + 5);
        __builtin_amdgcn_sched_barrier(0);
        step(y0, c0, kb + 2, kFull);
        fetch(y0, c0, kb + 6);
        __builtin_amdgcn_sched_barrier(0);
        step(y1, c1, kb + 3, kFull);
        fetch(y1, c1, kb + 7);
        __builtin_amdgcn_sched_barrier(0);
    }
    if (kb + 3 < nkb) {   // the last full group, refilling only what remains
        step(x0, b0, kb, kTail);
        if (kb + 4 < nkb) fetch(x0, b0, kb + 4);
        step(x1, b1, kb + 1, kTail);
        if (kb + 5 < nkb) fetch(x1, b1, kb + 5);
        step(y0, c0, kb + 2, kTail);
        if (kb + 6 < nkb) fetch(y0, c0, kb + 6);
        step(y1, c1, kb + 3, kTail);
        kb += 4;
    }
    if (kb < nkb) step(x0, b0, kb, kTail);
    if (kb + 1 < nkb) step(x1, b1, kb + 1, kTail);
    if (kb + 2 < nkb) step(y0, c0, kb + 2, kTail);
    // lane (r, g), value v of column block tb holds Z_2 column 16 tb + acc_row(g, v)
#pragma unroll
    for (int tb = 0; tb < NT; ++tb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const bool ok = 16 * tb + acc_row<T>(g, v) <= tlast;
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb) acc[pb][tb][v] = ok ? acc[pb][tb][v] : 0;
        }
}

// Last-core fragments of the reconstruction through a buffer resource of the
// core's exact size: rows past the rank lie beyond it and read as zero (their
// Z_2 columns are zero), so a fragment's byte offset is the lane's offset in
// step 0 plus a uniform stride per K step, kept in the range-checked vector
// offset, with no clamp.
template <typename T>
struct LastCoreReader {
    __amdgpu_buffer_rsrc_t rs;
    uint32_t nl, kstride;
    __device__ __forceinline__ LastCoreReader(const void* core, int rM, uint32_t n_last)
        : rs(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(core), (short)0,
                                               (int)((uint32_t)rM * n_last * (uint32_t)sizeof(T)), 0x00020000)),
          nl(n_last), kstride(4u * n_last * (uint32_t)sizeof(T)) {}
    __device__ __forceinline__ uint32_t lane(int g, uint32_t c) const { return ((uint32_t)g * nl + c) * (uint32_t)sizeof(T); }
    __device__ __forceinline__ T ld(int k, uint32_t vo) const {
        const uint32_t off = vo + (uint32_t)k * kstride;
        if constexpr (sizeof(T) == 8) return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b64(rs, off, 0, 0));
        else return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0));
    }
};

// Last product of a reconstruction wave tile: NPB row blocks of 16 rows,
// stored straight from the accumulators (lane (r, g), value v: row
// L0 + 16 pb + g + 4 v of column 16 cp + r, so that each store instruction
// writes 128-byte row segments).  The core fragments (lane (r, g) of step
// kb, block cp: G_3(4 kb + g, 16 cp + r)) run D steps ahead in a ring (N:
// steps 0 .. D-1 of a block, R: the later steps; the last D steps of a
// block fetch the first D of the next).
template <int NKB, int NPB, int D>
__device__ __forceinline__ void last_store_w(const TTArgs& a, int64_t i, int64_t L0, int r, int g,
                                             const double (&zf)[NPB][NKB]) {
    static_assert(D <= NKB, "ring deeper than a block");
    const int n_cb = (int)((a.n_last + 15) / 16);
    const LastCoreReader<double> lc(a.set[0].core[1], a.set[0].rM, (uint32_t)a.n_last);
    double* out = static_cast<double*>(a.out);
    const uint32_t nl = (uint32_t)a.n_last, clast = nl - 1;
    auto colc = [&](int cp) {
        const uint32_t c = (uint32_t)(16 * cp + r);
        return c < clast ? c : clast;
    };
    double N[D], R[D];
    uint32_t vo = lc.lane(g, colc(0));
#pragma unroll
    for (int s = 0; s < D; ++s) N[s] = lc.ld(s, vo);
    for (int cp = 0; cp < n_cb; ++cp) {
        const uint32_t von = lc.lane(g, colc(cp + 1 < n_cb ? cp + 1 : cp));
        double4_t acc[NPB];
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) acc[pb] = zero_accv<double4_t>();
        // MORE: a next block exists, whose first steps the last steps fetch
        // (one copy of the unrolled block each way, chosen once per block)
        auto block = [&](auto more) {
#pragma unroll
            for (int s = 0; s < NKB; ++s) {
                const double f = s < D ? N[s] : R[s % D];
#pragma unroll
                for (int pb = 0; pb < NPB; ++pb) acc[pb] = mfma(zf[pb][s], f, acc[pb]);
                const int k = s + D;
                if (k < NKB) R[k % D] = lc.ld(k, vo);
                else if constexpr (decltype(more)::value) N[k - NKB] = lc.ld(k - NKB, von);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        if (cp + 1 < n_cb) block(std::true_type{});
        else block(std::false_type{});
        const int64_t col = (int64_t)cp * 16 + r;
        if (col < a.n_last) {
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int64_t L = L0 + 16 * pb + g + 4 * v;
                    // where rows start on 128-byte lines, each instruction
                    // covers whole lines (16 lanes of one row) and is written
                    // around the caches; a partial line is not (measured:
                    // nontemporal partial lines cost several times more)
                    if (L < a.NL) {
                        double* dst = out + (L * a.n_mid + i) * a.n_last + col;
                        if (a.lines) __builtin_nontemporal_store(acc[pb][v], dst);
                        else *dst = acc[pb][v];
                    }
                }
        }
        vo = von;
    }
}

// FP64 reconstruction for d = 3 by wave tiles: a tile is 16 NPB rows of G_1
// for one middle index i (tile = i * ceil(n_1 / (16 NPB)) + row block, or
// row block * n_2 + i for short output rows, TTArgs::ifast), the
// interfaces Z_2 of its row blocks held in registers as the A fragments of
// the last product (the FP64 MFMA leaves value v of column block tb of Z_2
// in the lanes and order that the last product's K step 4 tb + v takes as
// its A operand).  The four waves of a workgroup, and consecutive
// workgroups of one XCD, share i and so the middle core slice in L2.  The
// core ring is 8 steps deep (4 for four row blocks, whose steps are twice
// as long).
template <int NKB, int NPB>
__global__ __launch_bounds__(256) void k_tt_wave(TTArgs a, int64_t ntiles) {
    constexpr int NT = (NKB + 3) / 4;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nLb = (a.NL + 16 * NPB - 1) / (16 * NPB);
    const int64_t wl = xcd_tile(gridDim.x);
    for (int64_t tile = wl * 4 + wave; tile < ntiles; tile += (int64_t)gridDim.x * 4) {
        const int64_t i = a.ifast ? tile % a.n_mid : tile / nLb;
        const int64_t L0 = (a.ifast ? tile / a.n_mid : tile % nLb) * 16 * NPB;
        double zf[NPB][NKB];
        {
            int ln = lane;
            asm volatile("" : "+v"(ln));
            double4_t acc[NPB][NT];
            middle_w_tile<double, NT, NPB>(a, a.set[0], i, L0, ln & 15, ln >> 4, acc);
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
                for (int tb = 0; tb < NT; ++tb)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (4 * tb + v < NKB) zf[pb][4 * tb + v] = acc[pb][tb][v];
        }
        int ln = lane;
        asm volatile("" : "+v"(ln));
        last_store_w<NKB, NPB, (NKB < (NPB == 4 ? 4 : 8) ? NKB : (NPB == 4 ? 4 : 8))>(a, i, L0, ln & 15, ln >> 4, zf);
    }
}

static void launch_wave(int nkb, int npb, dim3 grid, hipStream_t st, const TTArgs& a, int64_t ntiles) {
#define LRC_TW(K, P) hipLaunchKernelGGL((k_tt_wave<K, P>), grid, dim3(256), 0, st, a, ntiles)
#define LRC_TWK(K) \
    do {                                 \
        if (npb == 1) LRC_TW(K, 1);      \
        else if (npb == 4) LRC_TW(K, 4); \
        else LRC_TW(K, 2);               \
    } while (0)
    switch (nkb) {
    case 4: LRC_TWK(4); break;
    case 5: LRC_TWK(5); break;
    case 8: LRC_TWK(8); break;
    case 9: LRC_TWK(9); break;
    case 12: LRC_TWK(12); break;
    case 16: LRC_TWK(16); break;
    default: LRC_TWK(17); break;
    }
#undef LRC_TWK
#undef LRC_TW
}

// ---------------------------------------------------------------------------
// Quality of an FP64 reconstruction against its reference, fused into the
// wave tiles (Sec. sec:hyperspectral_application): the last product's
// values y = scale * T^(L, i, c) meet the reference X(L, i, c) while they
// are in registers, and nothing of the reconstruction is written.  Pixels
// are the rows (L, i), bands the columns c.
//   bands:  per 16-column block, each lane adds its elements' shifted sums
//           (shift s_c = X(0, c)), squares, cross products, squared
//           differences and squares of X, and its minimum and maximum; the
//           four lane groups of a column are combined in a fixed butterfly
//           and added into the wave's own LDS accumulators [QS_N][n_d];
//   pixels: each lane keeps the dot product and squared norms of its rows
//           over the tile's column blocks in registers; at the tile's end
//           they are added across the 16 column lanes and give the angles.
// At the end the workgroup adds its four waves in wave order into one
// partial per workgroup in the layout of the dense quality kernels, whose
// reductions finish the measures.
constexpr int kQualNpb = 2;   // row blocks per quality tile (register budget)

template <int NKB, int NPB, int D>
__device__ __forceinline__ void last_quality_w(const TTArgs& a, int64_t i, int64_t L0, int r, int g,
                                               const double (&zf)[NPB][NKB], const double* __restrict__ X,
                                               double scale, double* wacc, double (&pd)[NPB][4],
                                               double (&px)[NPB][4], double (&py)[NPB][4]) {
    static_assert(D <= NKB, "ring deeper than a block");
    const int n_cb = (int)((a.n_last + 15) / 16);
    const int64_t B = a.n_last;
    const LastCoreReader<double> lc(a.set[0].core[1], a.set[0].rM, (uint32_t)a.n_last);
    const uint32_t nl = (uint32_t)a.n_last, clast = nl - 1;
    auto colc = [&](int cp) {
        const uint32_t c = (uint32_t)(16 * cp + r);
        return c < clast ? c : clast;
    };
    int64_t prow[NPB][4];   // X offsets of the lane's rows (clamped), validity in rok
    bool rok[NPB][4];
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int64_t L = L0 + 16 * pb + g + 4 * v;
            rok[pb][v] = L < a.NL;
            prow[pb][v] = ((rok[pb][v] ? L : a.NL - 1) * a.n_mid + i) * B;
        }
    double N[D], R[D];
    uint32_t vo = lc.lane(g, colc(0));
#pragma unroll
    for (int s = 0; s < D; ++s) N[s] = lc.ld(s, vo);
    for (int cp = 0; cp < n_cb; ++cp) {
        const uint32_t von = lc.lane(g, colc(cp + 1 < n_cb ? cp + 1 : cp));
        const int64_t col = (int64_t)cp * 16 + r;
        const bool cok = col < B;
        const int64_t cc = cok ? col : B - 1;
        // the reference values of this block, in flight during its products
        double xv[NPB][4];
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
            for (int v = 0; v < 4; ++v) xv[pb][v] = X[prow[pb][v] + cc];
        const double sh = X[cc];
        __builtin_amdgcn_sched_barrier(0);
        double4_t acc[NPB];
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) acc[pb] = zero_accv<double4_t>();
        auto block = [&](auto more) {
#pragma unroll
            for (int s = 0; s < NKB; ++s) {
                const double f = s < D ? N[s] : R[s % D];
#pragma unroll
                for (int pb = 0; pb < NPB; ++pb) acc[pb] = mfma(zf[pb][s], f, acc[pb]);
                const int k = s + D;
                if (k < NKB) R[k % D] = lc.ld(k, vo);
                else if constexpr (decltype(more)::value) N[k - NKB] = lc.ld(k - NKB, von);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        if (cp + 1 < n_cb) block(std::true_type{});
        else block(std::false_type{});
        double st[QS_N];
#pragma unroll
        for (int q = 0; q < QS_MIN; ++q) st[q] = 0.0;
        st[QS_MIN] = sh;
        st[QS_MAX] = sh;
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const bool ok = cok && rok[pb][v];
                const double x = ok ? xv[pb][v] : 0.0, y = ok ? scale * acc[pb][v] : 0.0;
                pd[pb][v] += x * y;
                px[pb][v] += x * x;
                py[pb][v] += y * y;
                const double dx = ok ? x - sh : 0.0, dy = ok ? y - sh : 0.0, dd = x - y;
                st[QS_X] += dx;
                st[QS_Y] += dy;
                st[QS_XX] += dx * dx;
                st[QS_YY] += dy * dy;
                st[QS_XY] += dx * dy;
                st[QS_DD] += dd * dd;
                st[QS_X2] += x * x;
                if (ok) {
                    st[QS_MIN] = x < st[QS_MIN] ? x : st[QS_MIN];
                    st[QS_MAX] = x > st[QS_MAX] ? x : st[QS_MAX];
                }
            }
        // the four lane groups of this column: a fixed butterfly
#pragma unroll
        for (int off = 16; off <= 32; off <<= 1) {
#pragma unroll
            for (int q = 0; q < QS_MIN; ++q) st[q] += __shfl_xor(st[q], off, 64);
            const double mn = __shfl_xor(st[QS_MIN], off, 64), mx = __shfl_xor(st[QS_MAX], off, 64);
            st[QS_MIN] = mn < st[QS_MIN] ? mn : st[QS_MIN];
            st[QS_MAX] = mx > st[QS_MAX] ? mx : st[QS_MAX];
        }
        if (g == 0 && cok) {
#pragma unroll
            for (int q = 0; q < QS_MIN; ++q) wacc[q * B + col] += st[q];
            const double mn = wacc[QS_MIN * B + col], mx = wacc[QS_MAX * B + col];
            wacc[QS_MIN * B + col] = st[QS_MIN] < mn ? st[QS_MIN] : mn;
            wacc[QS_MAX * B + col] = st[QS_MAX] > mx ? st[QS_MAX] : mx;
        }
        vo = von;
    }
}

template <int NKB>
__global__ __launch_bounds__(256) void k_tt_wave_q(TTArgs a, int64_t ntiles, const double* __restrict__ X,
                                                   double scale, double* __restrict__ part,
                                                   double* __restrict__ part2) {
    constexpr int NPB = kQualNpb;
    constexpr int NT = (NKB + 3) / 4;
    constexpr int D = NKB < 8 ? NKB : 8;
    extern __shared__ double4_t smem_v[];
    __shared__ double wsam[4][2];
    double* qacc = reinterpret_cast<double*>(smem_v);   // [4 waves][QS_N][n_d]
    const int64_t B = a.n_last;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    double* wacc = qacc + (int64_t)wave * QS_N * B;
    for (int64_t c = lane; c < B; c += 64) {
        const double s = X[c];
#pragma unroll
        for (int q = 0; q < QS_MIN; ++q) wacc[q * B + c] = 0.0;
        wacc[QS_MIN * B + c] = s;
        wacc[QS_MAX * B + c] = s;
    }
    __syncthreads();
    const int64_t nLb = (a.NL + 16 * NPB - 1) / (16 * NPB);
    double asum = 0.0, cnt = 0.0;
    for (int64_t tile = (int64_t)blockIdx.x * 4 + wave; tile < ntiles; tile += (int64_t)gridDim.x * 4) {
        const int64_t i = tile / nLb;
        const int64_t L0 = (tile % nLb) * 16 * NPB;
        double zf[NPB][NKB];
        {
            int ln = lane;
            asm volatile("" : "+v"(ln));
            double4_t acc[NPB][NT];
            middle_w_tile<double, NT, NPB>(a, a.set[0], i, L0, ln & 15, ln >> 4, acc);
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
                for (int tb = 0; tb < NT; ++tb)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (4 * tb + v < NKB) zf[pb][4 * tb + v] = acc[pb][tb][v];
        }
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int r = ln & 15, g = ln >> 4;
        double pd[NPB][4], px[NPB][4], py[NPB][4];
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
            for (int v = 0; v < 4; ++v) pd[pb][v] = px[pb][v] = py[pb][v] = 0.0;
        last_quality_w<NKB, NPB, D>(a, i, L0, r, g, zf, X, scale, wacc, pd, px, py);
        // each row's sums over its 16 column lanes (fixed butterfly), then its angle
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
#pragma unroll
                for (int off = 1; off < 16; off <<= 1) {
                    pd[pb][v] += __shfl_xor(pd[pb][v], off, 64);
                    px[pb][v] += __shfl_xor(px[pb][v], off, 64);
                    py[pb][v] += __shfl_xor(py[pb][v], off, 64);
                }
                const int64_t L = L0 + 16 * pb + g + 4 * v;
                const double nn = __builtin_sqrt(px[pb][v]) * __builtin_sqrt(py[pb][v]);
                if (r == 0 && L < a.NL && nn > 0.0) {
                    double c = pd[pb][v] / nn;
                    c = c > 1.0 ? 1.0 : (c < -1.0 ? -1.0 : c);
                    asum += acos(c);
                    cnt += 1.0;
                }
            }
    }
    asum = wave_sum(asum);
    cnt = wave_sum(cnt);
    if (lane == 0) {
        wsam[wave][0] = asum;
        wsam[wave][1] = cnt;
    }
    __syncthreads();
    const int64_t blk = blockIdx.x;
    for (int64_t e = tid; e < QS_N * B; e += 256) {
        const int q = (int)(e / B);
        const double* w0 = qacc + e;
        double v = w0[0];
        for (int w = 1; w < 4; ++w) {
            const double o = w0[(int64_t)w * QS_N * B];
            v = q == QS_MIN ? (o < v ? o : v) : (q == QS_MAX ? (o > v ? o : v) : v + o);
        }
        part[blk * QS_N * B + e] = v;
    }
    if (tid == 0) {
        part2[2 * blk] = ((wsam[0][0] + wsam[1][0]) + wsam[2][0]) + wsam[3][0];
        part2[2 * blk + 1] = ((wsam[0][1] + wsam[1][1]) + wsam[2][1]) + wsam[3][1];
    }
}

// FP32 accumulators of the transposed middle product hold, in lane (r, g),
// value v, Z_2(L0 + r, 16 tb + 4 g + v): lane group g has the four K values
// of step kb = 4 tb + g.  The A fragment of the FP32 last product wants
// lane group g to hold K value g of each step 4 tb + v: a 4 x 4 transpose
// between the four 16-lane groups and the four values, done as a swap of
// the off-diagonal 2 x 2 blocks across the 32-lane halves followed by a
// transpose inside each block across neighbouring 16-lane rows (the gfx950
// lane swaps permlane32_swap and permlane16_swap).
__device__ __forceinline__ void swap32(float& x, float& y) {
    const auto p = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, y),
                                                    false, false);
    x = __builtin_bit_cast(float, (unsigned)p[0]);
    y = __builtin_bit_cast(float, (unsigned)p[1]);
}
__device__ __forceinline__ void swap16(float& x, float& y) {
    const auto p = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(unsigned, x), __builtin_bit_cast(unsigned, y),
                                                    false, false);
    x = __builtin_bit_cast(float, (unsigned)p[0]);
    y = __builtin_bit_cast(float, (unsigned)p[1]);
}
__device__ __forceinline__ void transpose_groups(float4_t& a) {
    float v0 = a[0], v1 = a[1], v2 = a[2], v3 = a[3];
    swap32(v0, v2);
    swap32(v1, v3);
    swap16(v0, v1);
    swap16(v2, v3);
    a = float4_t{v0, v1, v2, v3};
}

// Output of one 16 x 16 block of a reconstruction wave tile (lane (r, g)
// holding row L0 + 16 pb + r, columns cbase + 4 g .. + 3) in storage type T.
// Rows that allow it take one vector store per lane (TS false, the kernel
// variant for TTArgs::vec4).  Otherwise (TS: n_last not a multiple of 4, or
// a misaligned output) the block goes through the
// wave's own 16 x 17 LDS tile `stl`, so that each store instruction writes
// 16 consecutive elements of each of 4 rows instead of four scattered
// elements per lane.  The wavefront-scope fences keep the exchange in order
// (LDS operations of one wave complete in order).
template <typename T, int NPB, bool TS>
__device__ __forceinline__ void store_block(const TTArgs& a, float* stl, int64_t i, int64_t L0, int64_t cbase,
                                            int r, int g, const float4_t (&acc)[NPB]) {
    T* out = static_cast<T*>(a.out);
    if constexpr (!TS) {
        const int64_t c0 = cbase + 4 * g;
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) {
            const int64_t L = L0 + 16 * pb + r;
            if (L >= a.NL || c0 + 3 >= a.n_last) continue;
            T* dst = out + (L * a.n_mid + i) * a.n_last + c0;
            typedef T v4_t __attribute__((ext_vector_type(4)));
            *reinterpret_cast<v4_t*>(dst) = v4_t{(T)acc[pb][0], (T)acc[pb][1], (T)acc[pb][2], (T)acc[pb][3]};
        }
    } else {
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
        for (int v = 0; v < 4; ++v) stl[r * 17 + 4 * g + v] = acc[pb][v];
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        const int64_t col = cbase + r;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int rr = 4 * j + g;
            const float v = stl[rr * 17 + r];
            const int64_t L = L0 + 16 * pb + rr;
            if (L < a.NL && col < a.n_last) out[(L * a.n_mid + i) * a.n_last + col] = (T)v;
        }
    }
    }
}

// FP32 last product of a reconstruction wave tile, computed transposed
// (core fragment as A, so that lane (r, g), value v holds row L0 + 16 pb + r,
// column 16 cp + 4 g + v: four consecutive columns, stored as one 16-byte
// vector where the row allows it).  Core ring as in last_store_w.
template <int NKB, int NPB, int D, bool TS>
__device__ __forceinline__ void last_store_w32(const TTArgs& a, float* stl, int64_t i, int64_t L0, int r, int g,
                                               const float (&zf)[NPB][NKB]) {
    static_assert(D <= NKB, "ring deeper than a block");
    const int n_cb = (int)((a.n_last + 15) / 16);
    const LastCoreReader<float> lc(a.set[0].core[1], a.set[0].rM, (uint32_t)a.n_last);
    const uint32_t nl = (uint32_t)a.n_last, clast = nl - 1;
    auto colc = [&](int cp) {
        const uint32_t c = (uint32_t)(16 * cp + r);
        return c < clast ? c : clast;
    };
    float N[D], R[D];
    uint32_t vo = lc.lane(g, colc(0));
#pragma unroll
    for (int s = 0; s < D; ++s) N[s] = lc.ld(s, vo);
    for (int cp = 0; cp < n_cb; ++cp) {
        const uint32_t von = lc.lane(g, colc(cp + 1 < n_cb ? cp + 1 : cp));
        float4_t acc[NPB];
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) acc[pb] = zero_accv<float4_t>();
        // MORE: a next block exists, whose first steps the last steps fetch
        // (one copy of the unrolled block each way, chosen once per block)
        auto block = [&](auto more) {
#pragma unroll
            for (int s = 0; s < NKB; ++s) {
                const float f = s < D ? N[s] : R[s % D];
#pragma unroll
                for (int pb = 0; pb < NPB; ++pb) acc[pb] = mfma(f, zf[pb][s], acc[pb]);
                const int k = s + D;
                if (k < NKB) R[k % D] = lc.ld(k, vo);
                else if constexpr (decltype(more)::value) N[k - NKB] = lc.ld(k - NKB, von);
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        if (cp + 1 < n_cb) block(std::true_type{});
        else block(std::false_type{});
        store_block<float, NPB, TS>(a, stl, i, L0, (int64_t)cp * 16, r, g, acc);
        vo = von;
    }
}

// FP32 reconstruction for d = 3 by wave tiles (as k_tt_wave, with the
// accumulators of the middle product transposed into A-fragment order).
template <int NKB, int NPB, bool TS>
__global__ __launch_bounds__(256) void k_tt_wave32(TTArgs a, int64_t ntiles) {
    constexpr int NT = (NKB + 3) / 4;
    constexpr int D = NKB < 8 ? NKB : 8;
    __shared__ float st_tile[4][16 * 17];   // per wave: rows not fit for vector stores
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nLb = (a.NL + 16 * NPB - 1) / (16 * NPB);
    const int64_t wl = xcd_tile(gridDim.x);
    for (int64_t tile = wl * 4 + wave; tile < ntiles; tile += (int64_t)gridDim.x * 4) {
        const int64_t i = a.ifast ? tile % a.n_mid : tile / nLb;
        const int64_t L0 = (a.ifast ? tile / a.n_mid : tile % nLb) * 16 * NPB;
        float zf[NPB][NKB];
        {
            int ln = lane;
            asm volatile("" : "+v"(ln));
            float4_t acc[NPB][NT];
            middle_w_tile<float, NT, NPB>(a, a.set[0], i, L0, ln & 15, ln >> 4, acc);
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
                for (int tb = 0; tb < NT; ++tb) {
                    transpose_groups(acc[pb][tb]);
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (4 * tb + v < NKB) zf[pb][4 * tb + v] = acc[pb][tb][v];
                }
        }
        int ln = lane;
        asm volatile("" : "+v"(ln));
        last_store_w32<NKB, NPB, D, TS>(a, st_tile[wave], i, L0, ln & 15, ln >> 4, zf);
    }
}

static void launch_wave32(int nkb, int npb, dim3 grid, hipStream_t st, const TTArgs& a, int64_t ntiles) {
#define LRC_TW(K, P)                                                                              \
    do {                                                                                          \
        if (a.vec4) hipLaunchKernelGGL((k_tt_wave32<K, P, false>), grid, dim3(256), 0, st, a, ntiles); \
        else hipLaunchKernelGGL((k_tt_wave32<K, P, true>), grid, dim3(256), 0, st, a, ntiles);        \
    } while (0)
#define LRC_TWK(K) \
    do {                                 \
        if (npb == 1) LRC_TW(K, 1);      \
        else if (npb == 2) LRC_TW(K, 2); \
        else LRC_TW(K, 4);               \
    } while (0)
    switch (nkb) {
    case 4: LRC_TWK(4); break;
    case 5: LRC_TWK(5); break;
    case 8: LRC_TWK(8); break;
    case 9: LRC_TWK(9); break;
    case 12: LRC_TWK(12); break;
    case 16: LRC_TWK(16); break;
    default: LRC_TWK(17); break;
    }
#undef LRC_TWK
#undef LRC_TW
}

// FP16 wave tiles: K steps of 32, lane (r, g) supplying K values
// 8 g .. 8 g + 7 of row r (A) or column r (B) in one 16-byte fragment.
// Middle product (transposed, FP32 accumulation): A from the staged middle
// core [n_2][Rt][Kp2], B from the staged rows of G_1 [n_1][Kp2]; the
// accumulator of column block tb holds, in lane (r, g), value v,
// Z_2(L0 + r, 16 tb + 4 g + v).  Chains are two or three steps long, so the
// fragments of two steps are fetched at once.
template <int NT>
__device__ __forceinline__ void middle_w16(const TTArgs& a, const TTSet& S, int64_t i, int64_t L0, int r, int g,
                                           float4_t (&acc)[NT]) {
    const half_t* mid = static_cast<const half_t*>(S.st_mid) + i * S.Rt * S.Kp2;   // uniform
    const uint32_t moff = (uint32_t)(r * S.Kp2 + 8 * g) * 2u;
    const int64_t tstep = 16 * (int64_t)S.Kp2;   // next column block
    const int64_t row = (L0 + r < a.NL) ? L0 + r : a.NL - 1;
    const half_t* zr = static_cast<const half_t*>(S.st_left) + row * S.Kp2 + 8 * g;
    const int nkb = S.Kp2 / 32;
    auto cl = [nkb](int k) { return k < nkb ? k : nkb - 1; };
    auto af = [&](half8_t (&x)[NT], int kb) {
        const half_t* mk = mid + cl(kb) * 32;
#pragma unroll
        for (int tb = 0; tb < NT; ++tb) x[tb] = ld_off(reinterpret_cast<const half8_t*>(mk + tb * tstep), moff);
    };
    auto bf = [&](int kb) { return *reinterpret_cast<const half8_t*>(zr + cl(kb) * 32); };
#pragma unroll
    for (int tb = 0; tb < NT; ++tb) acc[tb] = zero_accv<float4_t>();
    half8_t x0[NT], x1[NT];
    af(x0, 0);
    af(x1, 1);
    half8_t b0 = bf(0), b1 = bf(1);
    auto step = [&](const half8_t (&x)[NT], half8_t b) {
#pragma unroll
        for (int tb = 0; tb < NT; ++tb) acc[tb] = mfma(x[tb], b, acc[tb]);
    };
    int kb = 0;
    for (; kb + 1 < nkb; kb += 2) {
        step(x0, b0);
        af(x0, kb + 2);
        b0 = bf(kb + 2);
        __builtin_amdgcn_sched_barrier(0);
        step(x1, b1);
        af(x1, kb + 3);
        b1 = bf(kb + 3);
        __builtin_amdgcn_sched_barrier(0);
    }
    if (kb < nkb) step(x0, b0);
}

// The FP16 middle products of all NPB row blocks of a tile (one middle index,
// so the same G_2 fragments): the NT x NKB2 A fragments are fetched once and
// kept, then each row block needs only its rows of G_1 (Kp2 <= 32 NKB2).
// EXACT: Kp2 == 32 NKB2, so no K step is skipped at run time (a skip lets
// the compiler sink the row loads down to their use, one wait each).
template <int NT, int NKB2, int NPB, bool EXACT, class OutF>
__device__ __forceinline__ void middle_w16_tile(const TTArgs& a, const TTSet& S, int64_t i, int64_t L0, int r, int g,
                                                OutF emit) {
    const half_t* mid = static_cast<const half_t*>(S.st_mid) + i * S.Rt * S.Kp2;   // uniform
    const uint32_t moff = (uint32_t)(r * S.Kp2 + 8 * g) * 2u;
    const int64_t tstep = 16 * (int64_t)S.Kp2;
    const int nkb = EXACT ? NKB2 : S.Kp2 / 32;   // <= NKB2
    half8_t x[NKB2][NT];
#pragma unroll
    for (int kb = 0; kb < NKB2; ++kb) {
        const half_t* mk = mid + (kb < nkb ? kb : nkb - 1) * 32;
#pragma unroll
        for (int tb = 0; tb < NT; ++tb) x[kb][tb] = ld_off(reinterpret_cast<const half8_t*>(mk + tb * tstep), moff);
    }
    auto rows = [&](int pb, half8_t (&b)[NKB2]) {
        const int64_t row = (L0 + 16 * pb + r < a.NL) ? L0 + 16 * pb + r : a.NL - 1;
        const half_t* zr = static_cast<const half_t*>(S.st_left) + row * S.Kp2 + 8 * g;
#pragma unroll
        for (int kb = 0; kb < NKB2; ++kb) b[kb] = *reinterpret_cast<const half8_t*>(zr + (kb < nkb ? kb : nkb - 1) * 32);
    };
    half8_t bc[NKB2], bn[NKB2];
    rows(0, bc);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int pb = 0; pb < NPB; ++pb) {
        if (pb + 1 < NPB) rows(pb + 1, bn);   // next row block's rows, fetched ahead
        // keep the prefetch ahead of this block's products (the scheduler
        // would otherwise sink each load down to its use)
        __builtin_amdgcn_sched_barrier(0);
        float4_t acc[NT];
#pragma unroll
        for (int tb = 0; tb < NT; ++tb) acc[tb] = zero_accv<float4_t>();
#pragma unroll
        for (int kb = 0; kb < NKB2; ++kb) {
            if (!EXACT && kb >= nkb) break;
#pragma unroll
            for (int tb = 0; tb < NT; ++tb) acc[tb] = mfma(x[kb][tb], bc[kb], acc[tb]);
        }
        emit(pb, acc);
#pragma unroll
        for (int kb = 0; kb < NKB2; ++kb) bc[kb] = bn[kb];
    }
}

// Round the FP32 accumulators of column blocks 2 kb and 2 kb + 1 to FP16 and
// regroup them into the A fragment of K step kb of the last product: lane
// group g needs Z_2(L0 + r, 32 kb + 8 g .. 8 g + 7), held as four values by
// each of lane groups 2 (g mod 2) and 2 (g mod 2) + 1 of block 2 kb + g / 2.
// With the values packed in pairs, a swap across the 32-lane halves and one
// across neighbouring 16-lane rows bring them into place.
__device__ __forceinline__ unsigned pack_h2(float lo, float hi) {
    typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(unsigned, h2_t{(half_t)lo, (half_t)hi});
}
__device__ __forceinline__ void swap32u(unsigned& x, unsigned& y) {
    const auto p = __builtin_amdgcn_permlane32_swap(x, y, false, false);
    x = p[0];
    y = p[1];
}
__device__ __forceinline__ void swap16u(unsigned& x, unsigned& y) {
    const auto p = __builtin_amdgcn_permlane16_swap(x, y, false, false);
    x = p[0];
    y = p[1];
}
__device__ __forceinline__ half8_t regroup16(const float4_t& X, const float4_t& Y) {
    unsigned xa = pack_h2(X[0], X[1]), xb = pack_h2(X[2], X[3]);
    unsigned ya = pack_h2(Y[0], Y[1]), yb = pack_h2(Y[2], Y[3]);
    swap32u(xa, ya);
    swap32u(xb, yb);
    swap16u(xa, ya);
    swap16u(xb, yb);
    typedef unsigned u4_t __attribute__((ext_vector_type(4)));
    return __builtin_bit_cast(half8_t, u4_t{xa, xb, ya, yb});
}

// FP16 last product of a reconstruction wave tile, computed transposed
// (core fragment as A): lane (r, g), value v holds row L0 + 16 pb + r,
// column 16 cp + 4 g + v (four consecutive columns, one 8-byte store where
// the row allows it).  Each core fragment is refetched for the next column
// block right after its use.
template <int NKB, int NPB, bool TS>
__device__ __forceinline__ void last_store_w16(const TTArgs& a, float* stl, int64_t i, int64_t L0, int r, int g,
                                               const half8_t (&zf)[NPB][NKB]) {
    const int n_cb = (int)((a.n_last + 15) / 16);
    const int Kp3 = a.set[0].Kp3;
    const half8_t* b0 = static_cast<const half8_t*>(a.set[0].st_last);   // [ncp][Kp3], 16-byte units
    uint32_t off = (uint32_t)(r * Kp3 + 8 * g) * 2u;
    const uint32_t cstep = 16u * (uint32_t)Kp3 * 2u;
    half8_t N[NKB];
#pragma unroll
    for (int s = 0; s < NKB; ++s) N[s] = ld_off(b0 + 4 * s, off);
    for (int cp = 0; cp < n_cb; ++cp) {
        const uint32_t offn = cp + 1 < n_cb ? off + cstep : off;
        float4_t acc[NPB];
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) acc[pb] = zero_accv<float4_t>();
#pragma unroll
        for (int s = 0; s < NKB; ++s) {
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb) acc[pb] = mfma(N[s], zf[pb][s], acc[pb]);
            N[s] = ld_off(b0 + 4 * s, offn);
        }
        store_block<half_t, NPB, TS>(a, stl, i, L0, (int64_t)cp * 16, r, g, acc);
        off = offn;
    }
}

// As last_store_w16 with the staged last core resident in LDS (rows of
// pitch ldp halves): the fragments are LDS reads, which do not wait for the
// output stores (global loads would, as loads and stores complete in order).
template <int NKB, int NPB, bool TS>
__device__ __forceinline__ void last_store_w16l(const TTArgs& a, float* stl, const half_t* Ls, int ldp, int64_t i,
                                                int64_t L0, int r, int g, const half8_t (&zf)[NPB][NKB]) {
    const int n_cb = (int)((a.n_last + 15) / 16);
    // two column blocks per step (twice the independent products), the
    // next step's fragments read from LDS before this step's products
    auto frags = [&](half8_t (&f)[2][NKB], int cp) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int c = cp + h < n_cb ? cp + h : n_cb - 1;
            const half_t* lrow = Ls + (16 * c + r) * ldp + 8 * g;
#pragma unroll
            for (int s2 = 0; s2 < NKB; ++s2) f[h][s2] = *reinterpret_cast<const half8_t*>(lrow + 32 * s2);
        }
    };
    half8_t f[2][NKB], fn[2][NKB];
    frags(f, 0);
    for (int cp = 0; cp < n_cb; cp += 2) {
        if (cp + 2 < n_cb) frags(fn, cp + 2);
        float4_t acc[2][NPB];
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb) acc[h][pb] = zero_accv<float4_t>();
#pragma unroll
        for (int s2 = 0; s2 < NKB; ++s2)
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int pb = 0; pb < NPB; ++pb) acc[h][pb] = mfma(f[h][s2], zf[pb][s2], acc[h][pb]);
        if (!TS && a.vec8 && cp + 1 < n_cb) {
            // the two blocks' 32 columns regrouped so that lane (r, g) holds
            // columns 8 g .. 8 g + 7: one 16-byte store per row block, 64
            // bytes per row and instruction
            half_t* out = static_cast<half_t*>(a.out);
            const int64_t c0 = (int64_t)cp * 16 + 8 * g;
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb) {
                const half8_t v = regroup16(acc[0][pb], acc[1][pb]);
                const int64_t L = L0 + 16 * pb + r;
                if (L < a.NL && c0 + 8 <= a.n_last)
                    *reinterpret_cast<half8_t*>(out + (L * a.n_mid + i) * a.n_last + c0) = v;
            }
        } else {
            store_block<half_t, NPB, TS>(a, stl, i, L0, (int64_t)cp * 16, r, g, acc[0]);
            if (cp + 1 < n_cb) store_block<half_t, NPB, TS>(a, stl, i, L0, (int64_t)(cp + 1) * 16, r, g, acc[1]);
        }
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int s2 = 0; s2 < NKB; ++s2) f[h][s2] = fn[h][s2];
    }
}

// LDSB: the staged last core [ncp][Kp3] is first copied into LDS at pitch
// Kp3 + 8 halves (16-byte fragment reads of 16 rows fall on distinct banks).
// kW16 waves share one workgroup and its copy of the last core (8 and 16
// measured no faster than 4 on a 512 x 512 x 224 train).
constexpr int kW16 = 4;

template <int NKB, int NPB, bool LDSB, bool TS>
__global__ __launch_bounds__(64 * kW16) void k_tt_wave16(TTArgs a, int64_t ntiles) {
    constexpr int NT = 2 * NKB;
    extern __shared__ double4_t smem_v[];
    __shared__ float st_tile[kW16][16 * 17];   // per wave: rows not fit for vector stores
    half_t* Ls = reinterpret_cast<half_t*>(smem_v);
    const int ldp = a.set[0].Kp3 + 8;
    if constexpr (LDSB) {
        // every thread issues all of its loads (at most 16 chunks: the copy
        // is at most 64 KB) before the first LDS write, so the copy costs one
        // load latency instead of one per chunk
        typedef unsigned u4_t __attribute__((ext_vector_type(4)));
        const u4_t* src = static_cast<const u4_t*>(a.set[0].st_last);   // rows of Kp3 / 8 chunks
        const int cpr = a.set[0].Kp3 / 8, nch = a.ncp * cpr;
        constexpr int kMaxChunks = 65536 / 16 / (64 * kW16);
        u4_t buf[kMaxChunks];
#pragma unroll
        for (int q = 0; q < kMaxChunks; ++q) {
            const int idx = threadIdx.x + 64 * kW16 * q;
            if (idx < nch) buf[q] = src[idx];
        }
#pragma unroll
        for (int q = 0; q < kMaxChunks; ++q) {
            const int idx = threadIdx.x + 64 * kW16 * q;
            if (idx < nch) {
                const int row = idx / cpr, ch = idx - row * cpr;
                *reinterpret_cast<u4_t*>(Ls + row * ldp + 8 * ch) = buf[q];
            }
        }
        __syncthreads();
    }
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nLb = (a.NL + 16 * NPB - 1) / (16 * NPB);
    const int64_t wl = xcd_tile(gridDim.x);
    for (int64_t tile = wl * kW16 + wave; tile < ntiles; tile += (int64_t)gridDim.x * kW16) {
        const int64_t i = a.ifast ? tile % a.n_mid : tile / nLb;
        const int64_t L0 = (a.ifast ? tile / a.n_mid : tile % nLb) * 16 * NPB;
        half8_t zf[NPB][NKB];
        auto keep = [&](int pb, float4_t (&acc)[NT]) {
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) zf[pb][kb] = regroup16(acc[2 * kb], acc[2 * kb + 1]);
        };
        if (a.set[0].Kp2 == 32 * NKB) {
            // every row block's middle product from one fetch of the G_2 fragments
            int ln = lane;
            asm volatile("" : "+v"(ln));
            middle_w16_tile<NT, NKB, NPB, true>(a, a.set[0], i, L0, ln & 15, ln >> 4, keep);
        } else if (a.set[0].Kp2 <= 32 * 3) {
            int ln = lane;
            asm volatile("" : "+v"(ln));
            middle_w16_tile<NT, 3, NPB, false>(a, a.set[0], i, L0, ln & 15, ln >> 4, keep);
        } else {
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb) {
                int ln = lane;
                asm volatile("" : "+v"(ln));
                float4_t acc[NT];
                middle_w16<NT>(a, a.set[0], i, L0 + 16 * pb, ln & 15, ln >> 4, acc);
#pragma unroll
                for (int kb = 0; kb < NKB; ++kb) zf[pb][kb] = regroup16(acc[2 * kb], acc[2 * kb + 1]);
            }
        }
        int ln = lane;
        asm volatile("" : "+v"(ln));
        if constexpr (LDSB) last_store_w16l<NKB, NPB, TS>(a, st_tile[wave], Ls, ldp, i, L0, ln & 15, ln >> 4, zf);
        else last_store_w16<NKB, NPB, TS>(a, st_tile[wave], i, L0, ln & 15, ln >> 4, zf);
    }
}

// ---------------------------------------------------------------------------
// FP16 wave tiles reading the cores in place (d >= 3, no staging launch):
//   - the last core's rows G_d(t, :) go to LDS as they lie in memory (rows
//     t < Kp3 at pitch ldc = ncp + 16 halves, zero past r_{d-1}), and the
//     last product takes its operand (eight consecutive t for one column c)
//     with the transposing LDS read ds_read_b64_tr_b16;
//   - the middle core's operand (eight consecutive s for one t) is gathered
//     from the core in global memory: the tiles of one middle index run
//     consecutively, so its slice is found in the L2; columns t past r_{d-1}
//     are zero;
//   - the rows of G_1 (or of the left interface) are read as eight values
//     each, zero past r_{d-2}.
// WIDE: the middle product runs three K steps of 32 (Kp2 <= 96); else NKB
// (Kp2 <= 32 NKB).
__device__ __forceinline__ half8_t frag_krows16(const half_t* S, int ld, int rbase, int k0, int lane) {
    typedef short s4_t __attribute__((ext_vector_type(4)));
    typedef short s8_t __attribute__((ext_vector_type(8)));
    const int s = lane & 15;
    const half_t* p = S + (k0 + (s >> 2)) * ld + rbase + 4 * (s & 3);
    const s4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4_t*)(p));
    const s4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4_t*)(p + 4 * ld));
    const s8_t both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(half8_t, both);
}

template <int NKB, int NPB, bool WIDE, bool TS>
__global__ __launch_bounds__(64 * kW16) void k_tt_wave16d(TTArgs a, int64_t ntiles) {
    constexpr int NT = 2 * NKB;
    constexpr int NKB2 = WIDE ? 3 : NKB;
    extern __shared__ double4_t smem_v[];
    __shared__ float st_tile[kW16][16 * 17];   // per wave: rows not fit for vector stores
    half_t* Ls = reinterpret_cast<half_t*>(smem_v);
    const TTSet& S = a.set[0];
    const int rL = S.rL, rM = S.rM, Kp3 = S.Kp3;
    const int ldc = a.ncp + 16;
    {
        // G_d rows t < Kp3 into LDS, 16-byte chunks of eight columns (whole
        // aligned loads when the rows allow it, else eight scalar loads);
        // rows past r_{d-1} and columns past n_d are zero
        const half_t* g3 = static_cast<const half_t*>(S.core[1]);
        const int cpr = a.ncp / 8, nch = Kp3 * cpr;
        const bool vec = (a.n_last % 8 == 0) && (reinterpret_cast<uintptr_t>(g3) % 16 == 0);
        for (int c0 = threadIdx.x; c0 < nch; c0 += 8 * 64 * kW16) {
            half8_t buf[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int idx = c0 + 64 * kW16 * q;
                const int t = idx / cpr, c = 8 * (idx - (idx / cpr) * cpr);
                half8_t w;
#pragma unroll
                for (int j = 0; j < 8; ++j) w[j] = half_t(0);
                if (idx < nch && t < rM && c < a.n_last) {
                    const half_t* src = g3 + (int64_t)t * a.n_last + c;
                    if (vec) {
                        w = *reinterpret_cast<const half8_t*>(src);
                    } else {
#pragma unroll
                        for (int j = 0; j < 8; ++j) w[j] = c + j < a.n_last ? src[j] : half_t(0);
                    }
                }
                buf[q] = w;
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int idx = c0 + 64 * kW16 * q;
                if (idx < nch) {
                    const int t = idx / cpr, c = 8 * (idx - (idx / cpr) * cpr);
                    *reinterpret_cast<half8_t*>(Ls + t * ldc + c) = buf[q];
                }
            }
        }
        __syncthreads();
    }
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nLb = (a.NL + 16 * NPB - 1) / (16 * NPB);
    const int64_t wl = xcd_tile(gridDim.x);
    const half_t* g2 = static_cast<const half_t*>(S.core[0]);
    const half_t* g1 = static_cast<const half_t*>(S.core[2]);
    const int64_t ld2 = a.n_mid * (int64_t)rM;   // between consecutive s of G_{d-1}
    for (int64_t tile = wl * kW16 + wave; tile < ntiles; tile += (int64_t)gridDim.x * kW16) {
        const int64_t i = tile / nLb;
        const int64_t L0 = (tile % nLb) * 16 * NPB;
        int ln = lane;
        asm volatile("" : "+v"(ln));
        const int r = ln & 15, g = ln >> 4;
        // middle-core operands: lane (r, g) of step kb, block tb holds
        // G_{d-1}(32 kb + 8 g + j, i, 16 tb + r), j = 0..7
        half8_t x[NKB2][NT];
        const half_t* g2i = g2 + i * rM;
#pragma unroll
        for (int tb = 0; tb < NT; ++tb) {
            const int t = 16 * tb + r;
            const bool tok = t < rM;
            const int tc = tok ? t : rM - 1;
#pragma unroll
            for (int kb = 0; kb < NKB2; ++kb)
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int sv = 32 * kb + 8 * g + j;
                    const half_t v = g2i[(int64_t)(sv < rL ? sv : rL - 1) * ld2 + tc];
                    x[kb][tb][j] = tok ? v : half_t(0);
                }
        }
        auto rows = [&](int pb, half8_t (&b)[NKB2]) {
            const int64_t L = L0 + 16 * pb + r;
            const half_t* zr = g1 + (L < a.NL ? L : a.NL - 1) * rL;
#pragma unroll
            for (int kb = 0; kb < NKB2; ++kb)
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    const int sv = 32 * kb + 8 * g + j;
                    const half_t v = zr[sv < rL ? sv : rL - 1];
                    b[kb][j] = sv < rL ? v : half_t(0);
                }
        };
        half8_t zf[NPB][NKB];
        half8_t bc[NKB2], bn[NKB2];
        rows(0, bc);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb) {
            if (pb + 1 < NPB) rows(pb + 1, bn);
            __builtin_amdgcn_sched_barrier(0);
            float4_t acc[NT];
#pragma unroll
            for (int tb = 0; tb < NT; ++tb) acc[tb] = zero_accv<float4_t>();
#pragma unroll
            for (int kb = 0; kb < NKB2; ++kb)
#pragma unroll
                for (int tb = 0; tb < NT; ++tb) acc[tb] = mfma(x[kb][tb], bc[kb], acc[tb]);
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) zf[pb][kb] = regroup16(acc[2 * kb], acc[2 * kb + 1]);
#pragma unroll
            for (int kb = 0; kb < NKB2; ++kb) bc[kb] = bn[kb];
        }
        // last product: two column blocks per step, operands by transposing LDS reads
        const int n_cb = (int)((a.n_last + 15) / 16);
        auto frags = [&](half8_t (&f)[2][NKB], int cp) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int c = cp + h < n_cb ? cp + h : n_cb - 1;
#pragma unroll
                for (int s2 = 0; s2 < NKB; ++s2) f[h][s2] = frag_krows16(Ls, ldc, 16 * c, 32 * s2 + 8 * g, ln);
            }
        };
        half8_t f[2][NKB], fn[2][NKB];
        frags(f, 0);
        for (int cp = 0; cp < n_cb; cp += 2) {
            if (cp + 2 < n_cb) frags(fn, cp + 2);
            float4_t acc[2][NPB];
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int pb = 0; pb < NPB; ++pb) acc[h][pb] = zero_accv<float4_t>();
#pragma unroll
            for (int s2 = 0; s2 < NKB; ++s2)
#pragma unroll
                for (int h = 0; h < 2; ++h)
#pragma unroll
                    for (int pb = 0; pb < NPB; ++pb) acc[h][pb] = mfma(f[h][s2], zf[pb][s2], acc[h][pb]);
            if (!TS && a.vec8 && cp + 1 < n_cb) {
                half_t* out = static_cast<half_t*>(a.out);
                const int64_t c0 = (int64_t)cp * 16 + 8 * g;
#pragma unroll
                for (int pb = 0; pb < NPB; ++pb) {
                    const half8_t v = regroup16(acc[0][pb], acc[1][pb]);
                    const int64_t L = L0 + 16 * pb + r;
                    if (L < a.NL && c0 + 8 <= a.n_last)
                        *reinterpret_cast<half8_t*>(out + (L * a.n_mid + i) * a.n_last + c0) = v;
                }
            } else {
                store_block<half_t, NPB, TS>(a, st_tile[wave], i, L0, (int64_t)cp * 16, r, g, acc[0]);
                if (cp + 1 < n_cb)
                    store_block<half_t, NPB, TS>(a, st_tile[wave], i, L0, (int64_t)(cp + 1) * 16, r, g, acc[1]);
            }
#pragma unroll
            for (int h = 0; h < 2; ++h)
#pragma unroll
                for (int s2 = 0; s2 < NKB; ++s2) f[h][s2] = fn[h][s2];
        }
    }
}

// The in-place kernel serves three-core FP16 trains (and trains of more
// cores whose two last cores are merged: 16^6 at ranks 9-25, 2048 tiles,
// 20.5 against 23.8 us with sides, staging and kernel) whose middle product
// has at most three K steps, whose last product at most two (three hold 259
// VGPRs, one wave per SIMD) and whose last core fits 64 KB of LDS at its
// pitch, when they have at most 2048 tiles: there the staging launch weighs
// most, while with more tiles the gathered middle-core operands of each tile
// cost more than the copy saves.  Measured with rocprofv3, in place against
// staged copy + kernel: 145 x 145 x 200 at rank 36 10.4 against 15.5 us,
// 256^3 at rank 15 11.9 against 14.8 us; 512 x 512 x 224 at rank 33 (4096
// tiles) 37.5 against 38.6 us; at rank 65 (three K steps) 66.6 against
// 41.3 us; the 16^6 train (16384 tiles, rows of its left interface read as
// eight scalar values each) 39.4 against 32 us; and in the resident timing
// grid 512 x 217 x 204 and 610 x 340 x 103 (3472 and 3400 tiles) lost 6 us.
// Unmerged trains of four and more cores keep the staged kernel.
static size_t wave16d_lds(const TTPlan& p) {
    return (size_t)p.set[0].Kp3 * (round_up(p.n_last, 32) + 16) * sizeof(half_t);
}
static bool wave16d_ok(const TTPlan& p) {
    return p.prec == P16 && p.nsets == 1 && (p.d == 3 || p.mid == p.d - 3) && p.wave_nkb && p.wave_nkb <= 2 && p.set[0].Kp2 <= 96 &&
           p.wave_tiles <= 2048 && wave16d_lds(p) <= 65536;
}
static void launch_wave16d(const TTPlan& p, dim3 grid, hipStream_t st, const TTArgs& a, int64_t ntiles) {
    const size_t lds = wave16d_lds(p);
    const bool wide = p.set[0].Kp2 > 32 * p.wave_nkb;
#define LRC_TD(K, P, W)                                                                                            \
    do {                                                                                                           \
        if (a.vec4) hipLaunchKernelGGL((k_tt_wave16d<K, P, W, false>), grid, dim3(64 * kW16), lds, st, a, ntiles); \
        else hipLaunchKernelGGL((k_tt_wave16d<K, P, W, true>), grid, dim3(64 * kW16), lds, st, a, ntiles);         \
    } while (0)
#define LRC_TDW(K, P)             \
    do {                          \
        if (wide) LRC_TD(K, P, true); \
        else LRC_TD(K, P, false); \
    } while (0)
#define LRC_TDK(K)                          \
    do {                                    \
        if (p.wave_npb == 1) LRC_TDW(K, 1); \
        else if (p.wave_npb == 2) LRC_TDW(K, 2); \
        else LRC_TDW(K, 4);                 \
    } while (0)
    if (p.wave_nkb == 1) LRC_TDK(1);
    else LRC_TDK(2);
#undef LRC_TDK
#undef LRC_TDW
#undef LRC_TD
}

// The last core goes to LDS when it fits 64 KB at the padded pitch.
static void launch_wave16(int nkb, int npb, dim3 grid, hipStream_t st, const TTArgs& a, int64_t ntiles) {
    const size_t lds = (size_t)a.ncp * (a.set[0].Kp3 + 8) * sizeof(half_t);
    const bool in_lds = lds <= 65536;
#define LRC_TW(K, P)                                                                                  \
    do {                                                                                              \
        if (in_lds && a.vec4)                                                                         \
            hipLaunchKernelGGL((k_tt_wave16<K, P, true, false>), grid, dim3(64 * kW16), lds, st, a, ntiles);  \
        else if (in_lds)                                                                              \
            hipLaunchKernelGGL((k_tt_wave16<K, P, true, true>), grid, dim3(64 * kW16), lds, st, a, ntiles);   \
        else if (a.vec4)                                                                              \
            hipLaunchKernelGGL((k_tt_wave16<K, P, false, false>), grid, dim3(64 * kW16), 0, st, a, ntiles);   \
        else hipLaunchKernelGGL((k_tt_wave16<K, P, false, true>), grid, dim3(64 * kW16), 0, st, a, ntiles);   \
    } while (0)
#define LRC_TWK(K) \
    do {                                 \
        if (npb == 1) LRC_TW(K, 1);      \
        else if (npb == 2) LRC_TW(K, 2); \
        else LRC_TW(K, 4);               \
    } while (0)
    switch (nkb) {
    case 1: LRC_TWK(1); break;
    case 2: LRC_TWK(2); break;
    default: LRC_TWK(3); break;
    }
#undef LRC_TWK
#undef LRC_TW
}

// Workgroups of the wave-tile kernels: four tiles each (kW16 for FP16), at
// most 4096.
static int64_t wave_grid(const TTPlan& p) {
    const int w = p.prec == P16 ? kW16 : 4;
    return xcd_grid(std::min<int64_t>((p.wave_tiles + w - 1) / w, 4096));
}

// The certificate split by what its sums couple: set 0 (the base train)
// only meets T (sums 0 and 4), sets 1 and 2 (the augmented train in FP64 and
// as stored) meet T and each other (sums 1, 2, 3).  Each part runs as
// NPB-row-block wave tiles like the reconstruction, so every G_3 fragment
// feeds NS NPB products and every G_2 fragment NPB.  Last products of the NS
// sets for a tile, with T read once per column block before its products;
// the core ring runs D steps ahead as in last_store_w.
// NS = 3: all three sets in one pass over T (sums 0 .. 4).
template <int NS>
struct CertSets {
    static constexpr int nsum = NS == 1 ? 2 : (NS == 2 ? 3 : 5);
    __host__ __device__ static constexpr int set(int q) { return NS == 1 ? 0 : (NS == 2 ? 1 + q : q); }
};

template <int NKB, int NPB, int NS, int D>
__device__ __forceinline__ void last_cert_s(const TTArgs& a, const double* __restrict__ Tref, int64_t i, int64_t L0,
                                            int r, int g, const double (&zf)[NS][NPB][NKB],
                                            double (&sum)[CertSets<NS>::nsum]) {
    static_assert(D <= NKB, "ring deeper than a block");
    const int n_cb = (int)((a.n_last + 15) / 16);
    // G_3 of each set through a buffer resource of its exact size: rows past
    // the rank lie beyond it and read as zero (their Z_2 columns are zero), so
    // a fragment's byte offset is the lane's offset in step 0 plus a uniform
    // step stride, with no clamp
    __amdgpu_buffer_rsrc_t rs[NS];
#pragma unroll
    for (int q = 0; q < NS; ++q) {
        const TTSet& S = a.set[CertSets<NS>::set(q)];
        rs[q] = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(S.core[1]), (short)0,
                                                  (int)((uint32_t)S.rM * (uint32_t)a.n_last * 8u), 0x00020000);
    }
    const uint32_t nl = (uint32_t)a.n_last, clast = nl - 1, kstride = 32u * nl;   // 4 rows of 8 bytes
    auto colc = [&](int cp) {
        const uint32_t c = (uint32_t)(16 * cp + r);
        return c < clast ? c : clast;
    };
    auto bld = [&](int q, int k, uint32_t vo) {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(rs[q], vo + (uint32_t)k * kstride, 0, 0);
        return __builtin_bit_cast(double, v);
    };
    double N[D][NS], R[D][NS];
    uint32_t c = colc(0);
    uint32_t vo = ((uint32_t)g * nl + c) * 8u;
#pragma unroll
    for (int s = 0; s < D; ++s)
#pragma unroll
        for (int q = 0; q < NS; ++q) N[s][q] = bld(q, s, vo);
    for (int cp = 0; cp < n_cb; ++cp) {
        const uint32_t cn = colc(cp + 1 < n_cb ? cp + 1 : cp);
        const uint32_t von = ((uint32_t)g * nl + cn) * 8u;
        const int64_t col = (int64_t)cp * 16 + r;
        double tv[NPB][4];
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t L = L0 + 16 * pb + g + 4 * v;
                const bool ok = L < a.NL && col < a.n_last;
                tv[pb][v] = Tref[ok ? (L * a.n_mid + i) * a.n_last + col : 0];
            }
        double4_t acc[NS][NPB];
#pragma unroll
        for (int q = 0; q < NS; ++q)
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb) acc[q][pb] = zero_accv<double4_t>();
        auto block = [&](auto more) {
#pragma unroll
            for (int s = 0; s < NKB; ++s) {
#pragma unroll
                for (int q = 0; q < NS; ++q) {
                    const double f = s < D ? N[s][q] : R[s % D][q];
#pragma unroll
                    for (int pb = 0; pb < NPB; ++pb) acc[q][pb] = mfma(zf[q][pb][s], f, acc[q][pb]);
                }
                const int k = s + D;
#pragma unroll
                for (int q = 0; q < NS; ++q) {
                    if (k < NKB) R[k % D][q] = bld(q, k, vo);
                    else if constexpr (decltype(more)::value) N[k - NKB][q] = bld(q, k - NKB, von);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        if (cp + 1 < n_cb) block(std::true_type{});
        else block(std::false_type{});
#pragma unroll
        for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const bool ok = L0 + 16 * pb + g + 4 * v < a.NL && col < a.n_last;
                const double t = ok ? tv[pb][v] : 0.0;
                if constexpr (NS == 1) {
                    const double d0 = t - (ok ? acc[0][pb][v] : 0.0);
                    sum[0] += d0 * d0;
                    sum[1] += t * t;
                } else if constexpr (NS == 3) {
                    const double r0 = ok ? acc[0][pb][v] : 0.0, r1 = ok ? acc[1][pb][v] : 0.0;
                    const double r2 = ok ? acc[2][pb][v] : 0.0;
                    const double d0 = t - r0, d1 = t - r1, d2 = r1 - r2, d3 = t - r2;
                    sum[0] += d0 * d0;
                    sum[1] += d1 * d1;
                    sum[2] += d2 * d2;
                    sum[3] += d3 * d3;
                    sum[4] += t * t;
                } else {
                    const double r1 = ok ? acc[0][pb][v] : 0.0, r2 = ok ? acc[1][pb][v] : 0.0;
                    const double d1 = t - r1, d2 = r1 - r2, d3 = t - r2;
                    sum[0] += d1 * d1;
                    sum[1] += d2 * d2;
                    sum[2] += d3 * d3;
                }
            }
        vo = von;
    }
}

// One part of the split certificate (see last_cert_s): tiles of 16 NPB rows
// of G_1 for one middle index, ordered as in k_tt_wave.  Workgroup w writes
// its sums to part[row * G + w] (rows 0, 4 for NS = 1; 1, 2, 3 for NS = 2)
// and zeros to the entries w + gridDim.x, w + 2 gridDim.x, ... < G, so both
// parts fill the same [5][G] layout whatever their grids.
template <int NKB, int NPB, int NS>
__global__ __launch_bounds__(256) void k_tt_cert_s(TTArgs a, const double* __restrict__ Tref,
                                                   double* __restrict__ part, int64_t ntiles, int64_t G) {
    constexpr int NT = (NKB + 3) / 4;
    constexpr int NSUM = CertSets<NS>::nsum;
    constexpr int D = NKB < (NPB * NS >= 3 ? 4 : 8) ? NKB : (NPB * NS >= 3 ? 4 : 8);
    __shared__ double red[4][NSUM];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nLb = (a.NL + 16 * NPB - 1) / (16 * NPB);
    double sum[NSUM];
#pragma unroll
    for (int q = 0; q < NSUM; ++q) sum[q] = 0.0;
    const int64_t wl = xcd_tile(gridDim.x);
    for (int64_t tile = wl * 4 + wave; tile < ntiles; tile += (int64_t)gridDim.x * 4) {
        const int64_t i = a.ifast ? tile % a.n_mid : tile / nLb;
        const int64_t L0 = (a.ifast ? tile / a.n_mid : tile % nLb) * 16 * NPB;
        double zf[NS][NPB][NKB];
#pragma unroll
        for (int q = 0; q < NS; ++q) {
            int ln = lane;
            asm volatile("" : "+v"(ln));
            double4_t acc[NPB][NT];
            middle_w_tile<double, NT, NPB>(a, a.set[CertSets<NS>::set(q)], i, L0, ln & 15, ln >> 4, acc);
#pragma unroll
            for (int pb = 0; pb < NPB; ++pb)
#pragma unroll
                for (int tb = 0; tb < NT; ++tb)
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (4 * tb + v < NKB) zf[q][pb][4 * tb + v] = acc[pb][tb][v];
        }
        int ln = lane;
        asm volatile("" : "+v"(ln));
        last_cert_s<NKB, NPB, NS, D>(a, Tref, i, L0, ln & 15, ln >> 4, zf, sum);
    }
#pragma unroll
    for (int q = 0; q < NSUM; ++q) {
        const double w = wave_sum(sum[q]);
        if (lane == 0) red[wave][q] = w;
    }
    __syncthreads();
    if (threadIdx.x < NSUM) {
        const int row = NS == 1 ? (threadIdx.x == 0 ? 0 : 4) : (NS == 2 ? 1 + (int)threadIdx.x : (int)threadIdx.x);
        part[row * G + blockIdx.x] =
            ((red[0][threadIdx.x] + red[1][threadIdx.x]) + red[2][threadIdx.x]) + red[3][threadIdx.x];
        for (int64_t w = blockIdx.x + gridDim.x; w < G; w += gridDim.x) part[row * G + w] = 0.0;
    }
}

template <typename T>
static void launch_fused(int npb, int nlb, dim3 grid, size_t lds, hipStream_t st, const TTArgs& a) {
#define LRC_TT(P, L) hipLaunchKernelGGL((k_tt_fused<T, P, L>), grid, dim3(256), lds, st, a)
    switch (npb * 8 + nlb) {
    case 1 * 8 + 1: LRC_TT(1, 1); break;
    case 2 * 8 + 1: LRC_TT(2, 1); break;
    case 2 * 8 + 2: LRC_TT(2, 2); break;
    case 3 * 8 + 1: LRC_TT(3, 1); break;
    case 3 * 8 + 2: LRC_TT(3, 2); break;
    case 3 * 8 + 3: LRC_TT(3, 3); break;
    case 4 * 8 + 1: LRC_TT(4, 1); break;
    case 4 * 8 + 2: LRC_TT(4, 2); break;
    case 4 * 8 + 3: LRC_TT(4, 3); break;
    default: LRC_TT(4, 4); break;
    }
#undef LRC_TT
}

// ------------------------------------------------------------------- host --
// Tuning aids: LRC_TT_P (rows per tile: 16, 32 or 64) and LRC_TT_WGS (target
// workgroup count) override the defaults when set.
static int tune_env(const char* name, int dflt) {
    const char* e = std::getenv(name);
    if (!e) return dflt;
    const int v = std::atoi(e);
    return v > 0 ? v : dflt;
}
int plan_tt(TTPlan& p, const int64_t* dims, const int64_t* const* rank_sets, int nsets, int d, int prec,
            size_t max_lds, bool merge_right) {
    p = TTPlan{};
    p.d = d;
    p.prec = prec;
    p.nsets = nsets;
    for (int c = 0; c < d; ++c) p.dims[c] = dims[c];
    const int KB = mfma_kb(prec);
    const int e = elem_bytes(prec);
    const int acc_b = (prec == P64) ? 8 : 4;
    p.chain_rmax = 1;
    for (int q = 0; q < nsets; ++q) {
        for (int c = 0; c <= d; ++c) p.set[q].ranks[c] = rank_sets[q][c];
        if (d >= 4)
            for (int c = 1; c <= d - 2; ++c) p.chain_rmax = (int)std::max<int64_t>(p.chain_rmax, rank_sets[q][c]);
    }
    int kp3 = 0;
    // the three-core train with middle core `mid` (see TTPlan)
    auto set_train = [&](int mid) {
        p.mid = mid;
        p.n_mid = dims[mid];
        p.n_last = 1;
        for (int c = mid + 1; c < d; ++c) p.n_last *= dims[c];
        p.NL = 1;
        for (int c = 0; c < mid; ++c) p.NL *= dims[c];
        for (int q = 0; q < nsets; ++q) {
            TTPlanSet& s = p.set[q];
            s.rM = (int)rank_sets[q][mid + 1];
            s.rL = (int)rank_sets[q][mid];
            s.Kp2 = (int)round_up(s.rL, KB);
            s.Kp3 = (int)round_up(s.rM, KB);
            // LDS pitches: consecutive rows of a fragment read land on
            // different banks (one element of pad; 16 bytes for FP16 rows,
            // which are read 16 bytes at a time)
            const int pad = (prec == P16) ? 8 : 1;
            s.ldl = s.Kp2 + pad;
            s.ldf = s.Kp3 + pad;
            s.Rt = (int)round_up(s.rM, 16);
        }
        // the sets of one kernel share the K extent of the last product (their
        // chains run in step); the staged cores are zero beyond each rank
        kp3 = 0;
        for (int q = 0; q < nsets; ++q) kp3 = std::max(kp3, p.set[q].Kp3);
        for (int q = 0; q < nsets; ++q) {
            p.set[q].ldf += kp3 - p.set[q].Kp3;
            p.set[q].Kp3 = kp3;
        }
    };
    // Trains with a short last mode (rows of n_d e <= 128 bytes) take the two
    // last cores as one right core for the wave tiles, when its n_{d-1} n_d
    // columns stay within 4096 and the merged train still has 2048 tiles of
    // 16 rows (two waves per SIMD): the output rows become n_{d-1} times
    // longer and the left interface n_{d-2} times shorter (16^6 at ranks up
    // to 25: rows of 16 -> 256 entries, left interface 65536 -> 4096 rows).
    // LRC_TT_MERGE=0 never merges, =1 merges whenever the shapes allow.
    bool merge = merge_right && nsets == 1 && d >= 4 && dims[d - 2] * dims[d - 1] <= 4096;
    {
        int64_t nl = 1;
        for (int c = 0; c < d - 3; ++c) nl *= dims[c];
        const char* mv = std::getenv("LRC_TT_MERGE");
        if (mv && mv[0] == '0') merge = false;
        else if (!(mv && mv[0] == '1')) merge = merge && dims[d - 1] * e <= 128 && dims[d - 3] * ((nl + 15) / 16) >= 2048;
    }
    set_train(merge ? d - 3 : d - 2);
    // staged cores (layouts at TTSet); ncp covers whole pairs of column blocks
    auto stage_bytes = [&]() {
        size_t b = 0;
        const int64_t ncp = round_up(p.n_last, 32);
        for (int q = 0; q < nsets; ++q)
            b += (size_t)(round_up(p.n_mid * p.set[q].Rt * p.set[q].Kp2 * e, 256) +
                          round_up(ncp * p.set[q].Kp3 * e, 256));
        return b;
    };
    // With d = 3 the kernels run by wave tiles (k_tt_cert_s for the FP64
    // certificate, k_tt_wave / k_tt_wave32 / k_tt_wave16 for the
    // reconstruction) when the last product's K extent fits one of their
    // register layouts: NKB K steps of 4 (FP64, FP32: Kp3 = 4 NKB <= 68) or of
    // 32 (FP16: Kp3 = 32 NKB <= 96).  Every set then takes that extent and
    // the matching column blocks of the middle product.  LRC_TT_WAVE=0
    // selects the LDS tiles; LRC_TT_WAVE_NPB (1, 2 or 4) sets the row blocks
    // per reconstruction tile.
    const char* wv = std::getenv("LRC_TT_WAVE");
    const bool wave_kind = d >= 3 && !(wv && wv[0] == '0') &&
                           ((prec == P64 && (nsets == 1 || nsets == 3)) || (prec != P64 && nsets == 1));
    for (int attempt = 0; attempt < 2 && wave_kind; ++attempt) {
    if (attempt == 1) {
        if (p.mid == d - 2) break;
        set_train(d - 2);   // the merged train did not fit the wave tiles
    }
    bool wave_ok = true;
    // FP64 / FP32 wave tiles read G_2 and G_3 in place with 32-bit byte offsets
    for (int q = 0; q < nsets && wave_ok; ++q) {
        const TTPlanSet& ps = p.set[q];
        wave_ok = (double)ps.rL * p.n_mid * ps.rM * e < 4294967296.0 && (double)ps.rM * p.n_last * e < 4294967296.0;
        // mid >= 2: one workgroup per prefix forms the left interface, its
        // row vectors (ranks r_1 .. r_{mid-1}) in 2 x 32 KB of LDS
        int64_t npfx = 1;
        for (int c = 0; c <= p.mid - 2; ++c) npfx *= dims[c];
        for (int c = 1; c <= p.mid - 1 && wave_ok; ++c) wave_ok = rank_sets[q][c] * acc_b <= 32768;
        wave_ok = wave_ok && npfx < 2147483647;
    }
    if (wave_ok) {
        int nkb = 0;
        if (prec == P16) {
            if (kp3 <= 96) nkb = kp3 / 32;
        } else {
            // the certificate's kernel exists for the first list only; one set
            // (reconstruction) also has K extents 20 and 36 (ranks 17-20 and
            // 33-36, the paper's TT timing schedules) without padding
            static const int kNkb3[] = {4, 8, 12, 16, 17};
            static const int kNkb1[] = {4, 5, 8, 9, 12, 16, 17};
            const int* lst = nsets == 1 ? kNkb1 : kNkb3;
            const int cnt = nsets == 1 ? 7 : 5;
            for (int c = 0; c < cnt; ++c)
                if (4 * lst[c] >= kp3) {
                    nkb = lst[c];
                    break;
                }
        }
        if (nkb > 0) {
            for (int q = 0; q < nsets; ++q) {
                TTPlanSet& ps = p.set[q];
                if (prec == P16) {
                    ps.Kp3 = 32 * nkb;
                    ps.ldf = ps.Kp3 + 8;
                    ps.Rt = 32 * nkb;
                } else {
                    ps.Kp3 = 4 * nkb;
                    ps.ldf = ps.Kp3 + 1;
                    ps.Rt = 16 * ((nkb + 3) / 4);
                }
            }
            int npb = 1;
            if (nsets == 1) {
                // fewer row blocks per wave where the tiles would not give
                // every SIMD two waves (2048 tiles)
                int dflt = 4;
                while (dflt > 1 && p.n_mid * ((p.NL + 16 * dflt - 1) / (16 * dflt)) < 2048) dflt /= 2;
                npb = tune_env("LRC_TT_WAVE_NPB", dflt);
                if (npb != 1 && npb != 2 && npb != 4) npb = dflt;
            }
            p.wave_nkb = nkb;
            p.wave_npb = npb;
            p.BL = 16 * npb;
            p.BI = 1;
            p.P = 16 * npb;
            p.lds_bytes = 0;
            p.num_i_blocks = p.n_mid;
            p.num_L_blocks = (p.NL + p.BL - 1) / p.BL;
            p.grid_L = 1;
            p.wave_tiles = p.num_i_blocks * p.num_L_blocks;
            // FP16 stages its cores (K-contiguous fragments); FP64 / FP32 read them in place
            p.stage_bytes = prec == P16 ? stage_bytes() + (size_t)round_up(p.NL * p.set[0].Kp2 * e, 256) : 0;
            // the left interface of every set (mid >= 2) and the merged right
            // core (mid = d - 3), in the storage type
            for (int q = 0; q < nsets; ++q) {
                if (p.mid >= 2) p.stage_bytes += (size_t)round_up(p.NL * p.set[q].rL * e, 256);
                if (p.mid == d - 3) p.stage_bytes += (size_t)round_up(p.set[q].rM * p.n_last * e, 256);
            }
            return 0;
        }
    }
    }
    // the LDS tiles take the train as it is
    if (p.mid != d - 2) set_train(d - 2);
    // at most 64 KB of LDS per workgroup (80 KB for the three-set
    // certificate kernel), so that at least two workgroups share a compute
    // unit; a reconstruction whose buffers do not fit that takes the whole
    // LDS of the compute unit (160 KB on gfx950), one workgroup per unit
    // (the certificate falls back to dense reconstructions instead)
    const size_t lds_soft = nsets > 1 ? 81920 : 65536;
    const int P0 = tune_env("LRC_TT_P", (prec == P64) ? 32 : 64);
    for (int pass = 0; pass < (nsets == 1 ? 2 : 1) && p.P == 0; ++pass) {
    const size_t lds_cap = pass == 0 ? std::min(max_lds, lds_soft) : max_lds;
    for (int P = P0; P >= 16; P /= 2) {
        int BI, BL;
        if (d == 2) {
            BL = 1;
            BI = P;
        } else if (d >= 4 && p.n_mid <= P) {
            BI = (int)p.n_mid;       // every middle index: left rows are built once
            BL = std::max(1, P / BI);
        } else {
            BI = 1;
            BL = P;
        }
        if ((int64_t)BL > p.NL) BL = (int)std::max<int64_t>(1, p.NL);
        const int Peff = (int)round_up((int64_t)BL * BI, 16);
        const int BLpad = (int)round_up(BL, 16);
        if (Peff > 64 || BLpad > 64) continue;
        // one Z_{d-2} buffer, shared by the sets in turn; one Z_{d-1} per set
        size_t lds = 0, zl = 0;
        for (int q = 0; q < nsets; ++q) {
            zl = std::max<size_t>(zl, (size_t)round_up((int64_t)BLpad * p.set[q].ldl * e, 32));
            lds += (size_t)round_up((int64_t)Peff * p.set[q].ldf * e, 32);
        }
        lds += zl;
        if (d >= 4) lds += (size_t)2 * BL * p.chain_rmax * acc_b;
        if (lds <= lds_cap) {
            p.BL = BL;
            p.BI = BI;
            p.P = Peff;
            p.lds_bytes = lds;
            break;
        }
    }
    }
    if (p.P == 0) return -1;
    p.num_i_blocks = (p.n_mid + p.BI - 1) / p.BI;
    p.num_L_blocks = (p.NL + p.BL - 1) / p.BL;

    int64_t want = tune_env("LRC_TT_WGS", 4096) / std::max<int64_t>(1, p.num_i_blocks);
    if (want < 1) want = 1;
    if (want > p.num_L_blocks) want = p.num_L_blocks;
    if (want > 65535) want = 65535;
    p.grid_L = (int)want;
    p.stage_bytes = stage_bytes();
    return 0;
}

// Kernel arguments for the plan, with the cores of every set staged.
template <typename T>
static hipError_t prepare_tt(const TTPlan& p, const void* const* const* cores, void* out, Workspace& ws,
                             hipStream_t stream, const char* label, TTArgs& a) {
    a = TTArgs{};
    a.d = p.d;
    a.nsets = p.nsets;
    for (int c = 0; c < p.d; ++c) a.dims[c] = p.dims[c];
    for (int c = 0; c <= p.d - 3; ++c) {
        int64_t D = 1;
        for (int c2 = c + 1; c2 <= p.d - 3; ++c2) D *= p.dims[c2];
        a.divs[c] = D;
    }
    a.NL = p.NL;
    a.n_mid = p.n_mid;
    a.n_last = p.n_last;
    a.BL = p.BL;
    a.BI = p.BI;
    a.P = p.P;
    a.BLpad = (int)round_up(p.BL, 16);
    a.chain_rmax = p.chain_rmax;
    a.num_L_blocks = p.num_L_blocks;
    a.ncp = (int)round_up(p.n_last, 32);
    a.out = out;
    a.vec4 = out && (p.n_last % 4 == 0) && (reinterpret_cast<uintptr_t>(out) % (4 * sizeof(T)) == 0);
    a.vec8 = sizeof(T) == 2 && out && (p.n_last % 8 == 0) && (reinterpret_cast<uintptr_t>(out) % 16 == 0);
    a.lines = out && ((p.n_last * (int64_t)sizeof(T)) % 128 == 0) && (reinterpret_cast<uintptr_t>(out) % 128 == 0);
    // short output rows (n_d e < 1 KB): wave tiles of consecutive middle indices
    // write neighbouring segments of the same rows, so the rows fill up
    // together.  Not for FP16: its tiles of one middle index share the staged
    // G_{d-1} slice, which then stays in the L2 (512 x 512 x 224 at rank 65:
    // 40.7 -> 31.9 us; with 16-byte row stores the rows' locality matters less)
    a.ifast = p.wave_nkb && p.n_last * (int64_t)sizeof(T) < 1024 && sizeof(T) != 2;
    // the staging copy is timed under the kernel's label with a "_stage" suffix
    char stage_label[64];
    std::snprintf(stage_label, sizeof(stage_label), "%s_stage", label);
    // wave tiles of a train whose middle core is G_{mid+1}, mid >= 2: the left
    // interface of cores 1 .. mid takes the place of G_1; with mid = d - 3 the
    // merged right core takes the place of G_d (both formed here, timed with
    // the staging)
    const void* left[kTTMaxSets] = {};
    const void* right[kTTMaxSets] = {};
    if (p.wave_nkb && (p.mid >= 2 || p.mid == p.d - 3)) {
        KernelTimer ts(stage_label, stream);
        for (int q = 0; q < p.nsets; ++q) {
            LeftChain lc{};
            T* fin = nullptr;
            T* w = nullptr;
            size_t lds = 0;
            if (p.mid >= 2) {
                fin = static_cast<T*>(ws.take((size_t)p.NL * p.set[q].rL * sizeof(T)));
                if (ws.overrun || !fin) return hipErrorOutOfMemory;
                // the chain of cores 1 .. mid is the left chain of a train of mid + 2 cores
                lc.d = p.mid + 2;
                for (int c = 0; c < lc.d; ++c) {
                    lc.core[c] = cores[q][c];
                    lc.dims[c] = p.dims[c];
                }
                for (int c = 0; c <= lc.d; ++c) lc.ranks[c] = p.set[q].ranks[c];
                left_split(lc, sizeof(typename PrecTraits<T>::acc));
                lds = 2 * (size_t)lc.buf * sizeof(typename PrecTraits<T>::acc);
                left[q] = fin;
            }
            if (p.mid == p.d - 3) {
                lc.rtotal = p.set[q].rM * p.n_last;
                w = static_cast<T*>(ws.take((size_t)lc.rtotal * sizeof(T)));
                if (ws.overrun || !w) return hipErrorOutOfMemory;
                lc.ra = cores[q][p.d - 2];
                lc.rb = cores[q][p.d - 1];
                lc.rna = p.dims[p.d - 2];
                lc.rnb = p.dims[p.d - 1];
                lc.rru = p.set[q].ranks[p.d - 1];
                right[q] = w;
            }
            const int64_t blocks = lc.nleft + (lc.rtotal + 255) / 256;
            hipLaunchKernelGGL(k_tt_sides<T>, dim3((unsigned)blocks), dim3(256), lds, stream, lc, fin, w);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
    }
    // LDS: the shared Z_{d-2} buffer first, then one Z_{d-1} per set
    int off = 0;
    for (int q = 0; q < p.nsets; ++q)
        off = std::max(off, (int)round_up((int64_t)a.BLpad * p.set[q].ldl * (int64_t)sizeof(T), 32));
    for (int q = 0; q < p.nsets; ++q) {
        TTSet& S = a.set[q];
        const TTPlanSet& ps = p.set[q];
        S.core[0] = cores[q][p.mid];
        S.core[1] = right[q] ? right[q] : cores[q][p.d - 1];
        for (int c = 0; c <= p.d - 3; ++c) S.core[2 + c] = cores[q][c];
        if (left[q]) S.core[2] = left[q];   // wave tiles: G_1 of the equivalent three-core train
        for (int c = 0; c <= p.d; ++c) S.ranks[c] = ps.ranks[c];
        S.rL = ps.rL;
        S.rM = ps.rM;
        S.Kp2 = ps.Kp2;
        S.Kp3 = ps.Kp3;
        S.ldl = ps.ldl;
        S.ldf = ps.ldf;
        S.Rt = ps.Rt;
        S.zl_off = 0;
        S.zf_off = off;
        off += (int)round_up((int64_t)p.P * ps.ldf * (int64_t)sizeof(T), 32);
        S.st_mid = S.st_last = S.st_left = nullptr;
        if (p.wave_nkb && sizeof(T) >= 4) continue;   // the wave tiles read the cores in place
        if (sizeof(T) == 2 && wave16d_ok(p)) continue;  // so do these FP16 wave tiles
        {
            T* smid = static_cast<T*>(ws.take((size_t)p.n_mid * ps.Rt * ps.Kp2 * sizeof(T)));
            T* slast = static_cast<T*>(ws.take((size_t)a.ncp * ps.Kp3 * sizeof(T)));
            if (ws.overrun || !smid || !slast) return hipErrorOutOfMemory;
            // FP16 wave tiles also take the rows of G_1 at pitch Kp2
            const bool rows = sizeof(T) == 2 && p.wave_nkb;
            T* sl = nullptr;
            if (rows) {
                sl = static_cast<T*>(ws.take((size_t)p.NL * ps.Kp2 * sizeof(T)));
                if (ws.overrun || !sl) return hipErrorOutOfMemory;
            }
            const int64_t tmid = p.n_mid * ps.Rt * ps.Kp2, tlast = (int64_t)a.ncp * ps.Kp3;
            const int64_t trows = rows ? p.NL * ps.Kp2 : 0;
            const int64_t tot = tmid + tlast + trows;
            int64_t gs = (tot + 255) / 256;
            if (gs > 4096) gs = 4096;
            const bool narrow = tmid < 2147483647LL && tlast < 2147483647LL && trows < 2147483647LL;
            KernelTimer ts(stage_label, stream);
            if constexpr (sizeof(T) == 2) {
                if (rows && ps.Rt <= kStage16T && ps.Kp3 <= kStage16T && ps.rM <= kStage16T) {
                    const int64_t wg_mid = p.n_mid * (ps.Kp2 / 32), wg_last = a.ncp / 32;
                    const int64_t wg_rows = (p.NL * (ps.Kp2 / 8) + 255) / 256;
                    hipLaunchKernelGGL(k_stage16, dim3((unsigned)(wg_mid + wg_last + wg_rows)), dim3(256), 0, stream,
                                       (const half_t*)S.core[0], (const half_t*)S.core[1],
                                       (const half_t*)S.core[2], (half_t*)smid, (half_t*)slast, (half_t*)sl, p.n_mid,
                                       p.n_last, p.NL, ps.rL, ps.rM, ps.Kp2, ps.Kp3, ps.Rt, a.ncp, wg_mid, wg_last);
                    hipError_t e = hipGetLastError();
                    if (e != hipSuccess) return e;
                    S.st_mid = smid;
                    S.st_last = slast;
                    S.st_left = sl;
                    continue;
                }
            }
#define LRC_STAGE(IDX)                                                                                       \
    hipLaunchKernelGGL((k_stage<T, IDX>), dim3((unsigned)gs), dim3(256), 0, stream, (const T*)S.core[0], \
                       (const T*)S.core[1], rows ? (const T*)S.core[2] : (const T*)nullptr, smid, slast, sl, \
                       p.n_mid, p.n_last, p.NL, ps.rL, ps.rM, ps.rL, ps.Kp2, ps.Kp3, ps.Rt, a.ncp)
            if (narrow) LRC_STAGE(uint32_t);
            else LRC_STAGE(int64_t);
#undef LRC_STAGE
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            S.st_mid = smid;
            S.st_last = slast;
            S.st_left = sl;
        }
    }
    a.cb_off = off;
    return hipSuccess;
}

template <typename T>
static hipError_t tt_typed(const TTPlan& p, const void* const* const* cores, void* out, Workspace& ws,
                           hipStream_t stream, const char* label) {
    if (!label) label = p.prec == P64 ? "tt_fused_f64" : (p.prec == P32 ? "tt_fused_f32" : "tt_fused_f16");
    TTArgs a;
    hipError_t e = prepare_tt<T>(p, cores, out, ws, stream, label, a);
    if (e != hipSuccess) return e;
    if (p.wave_nkb) {
        KernelTimer tk(label, stream);
        const dim3 gw((unsigned)wave_grid(p));
        if constexpr (sizeof(T) == 8) launch_wave(p.wave_nkb, p.wave_npb, gw, stream, a, p.wave_tiles);
        else if constexpr (sizeof(T) == 4) launch_wave32(p.wave_nkb, p.wave_npb, gw, stream, a, p.wave_tiles);
        else if (wave16d_ok(p)) launch_wave16d(p, gw, stream, a, p.wave_tiles);
        else launch_wave16(p.wave_nkb, p.wave_npb, gw, stream, a, p.wave_tiles);
        return hipGetLastError();
    }
    dim3 grid((unsigned)p.num_i_blocks, (unsigned)p.grid_L);
    KernelTimer tk(label, stream);
    launch_fused<T>(p.P / 16, (int)round_up(p.BL, 16) / 16, grid, p.lds_bytes, stream, a);
    return hipGetLastError();
}

int64_t tt_cert_parts(const TTPlan& p) {
    return p.wave_nkb ? wave_grid(p) : p.num_i_blocks * (int64_t)p.grid_L;
}

hipError_t launch_tt_cert(const TTPlan& p, const void* const* const* cores, const double* Tref, double* part,
                          Workspace& ws, hipStream_t stream) {
    if (p.prec != P64 || p.nsets != 3 || p.P > 32) return hipErrorInvalidValue;
    TTArgs a;
    hipError_t e = prepare_tt<double>(p, cores, nullptr, ws, stream, "cert_tt_fused_f64", a);
    if (e != hipSuccess) return e;
    if (p.wave_nkb) {
        // the split certificate: set 0 with two row blocks per tile (one
        // where the tiles would not give every SIMD two waves), sets 1 and 2
        // together with one (two would exceed the registers of two waves per
        // SIMD), each part with the K steps of its own ranks
        const int64_t G = wave_grid(p);
        auto nkb_of = [](int rM) {
            static const int lst[] = {4, 8, 12, 16, 17};
            for (int c : lst)
                if (4 * c >= rM) return c;
            return 0;
        };
        const int nkA = nkb_of(p.set[0].rM), nkB = nkb_of(std::max(p.set[1].rM, p.set[2].rM));
        if (!nkA || !nkB) return hipErrorInvalidValue;
        auto tiles = [&](int npb) { return p.n_mid * ((p.NL + 16 * npb - 1) / (16 * npb)); };
        const int npA = tiles(2) >= 2048 ? 2 : 1;
        const int64_t ntA = tiles(npA), ntB = tiles(1);
        const dim3 gA(xcd_grid(std::min<int64_t>((ntA + 3) / 4, 4096))), gB(xcd_grid(std::min<int64_t>((ntB + 3) / 4, 4096)));
        if ((int64_t)gA.x > G || (int64_t)gB.x > G) return hipErrorInvalidValue;
        KernelTimer tk("cert_tt_fused_f64", stream);
#define LRC_TCS(K, P, S, g, nt) \
    hipLaunchKernelGGL((k_tt_cert_s<K, P, S>), g, dim3(256), 0, stream, a, Tref, part, nt, G)
#define LRC_TCS_K(P, S, nk, g, nt)                    \
    switch (nk) {                                     \
    case 4: LRC_TCS(4, P, S, g, nt); break;           \
    case 8: LRC_TCS(8, P, S, g, nt); break;           \
    case 12: LRC_TCS(12, P, S, g, nt); break;         \
    case 16: LRC_TCS(16, P, S, g, nt); break;         \
    default: LRC_TCS(17, P, S, g, nt); break;         \
    }
        // one pass over T with the three sets in each wave (default), or
        // (LRC_TT_CERT_SPLIT=1) the base set and the augmented pair as two
        // kernels that each read T
        static const bool split = [] {
            const char* e = std::getenv("LRC_TT_CERT_SPLIT");
            return e && e[0] == '1';
        }();
        if (!split) {
            const int nk = std::max(nkA, nkB);
            LRC_TCS_K(1, 3, nk, gB, ntB)
        } else {
            if (npA == 2) {
                LRC_TCS_K(2, 1, nkA, gA, ntA)
            } else {
                LRC_TCS_K(1, 1, nkA, gA, ntA)
            }
            LRC_TCS_K(1, 2, nkB, gB, ntB)
        }
#undef LRC_TCS_K
#undef LRC_TCS
        return hipGetLastError();
    }
    const dim3 grid((unsigned)p.num_i_blocks, (unsigned)p.grid_L);
    const int64_t nparts = tt_cert_parts(p);
    const int npb = p.P / 16, nlb = (int)round_up(p.BL, 16) / 16;
    KernelTimer tk("cert_tt_fused_f64", stream);
#define LRC_TTC(P, L) hipLaunchKernelGGL((k_tt_cert<P, L>), grid, dim3(256), p.lds_bytes, stream, a, Tref, part, nparts)
    // the three sets' accumulators fit the registers for tiles of up to 32 rows
    switch (npb * 8 + nlb) {
    case 1 * 8 + 1: LRC_TTC(1, 1); break;
    case 2 * 8 + 1: LRC_TTC(2, 1); break;
    case 2 * 8 + 2: LRC_TTC(2, 2); break;
    default: return hipErrorInvalidValue;
    }
#undef LRC_TTC
    return hipGetLastError();
}

hipError_t launch_tt(const TTPlan& p, const void* const* cores, void* out, Workspace& ws, hipStream_t stream,
                     const char* label) {
    const void* const* sets[1] = {cores};
    if (p.prec == P64) return tt_typed<double>(p, sets, out, ws, stream, label);
    if (p.prec == P32) return tt_typed<float>(p, sets, out, ws, stream, label);
    return tt_typed<half_t>(p, sets, out, ws, stream, label);
}

static size_t quality_lds(int64_t B) { return (size_t)4 * QS_N * B * sizeof(double); }

int64_t tt_quality_blocks(const TTPlan& p, size_t max_lds) {
    // the measures index the last mode's bands: the train as it is
    if (p.prec != P64 || p.nsets != 1 || !p.wave_nkb || p.mid != p.d - 2) return 0;
    const size_t lds = quality_lds(p.n_last);
    if (lds > max_lds || lds > 131072) return 0;
    const int64_t per_cu = std::max<int64_t>(1, (int64_t)(163840 / lds));
    const int64_t tiles = p.n_mid * ((p.NL + 16 * kQualNpb - 1) / (16 * kQualNpb));
    return std::max<int64_t>(1, std::min<int64_t>((tiles + 3) / 4, 256 * per_cu));
}

hipError_t launch_tt_quality(const TTPlan& p, const void* const* cores, const double* X, double scale,
                             double* part, double* part2, size_t max_lds, Workspace& ws, hipStream_t stream) {
    const int64_t G = tt_quality_blocks(p, max_lds);
    if (!G) return hipErrorInvalidValue;
    TTArgs a;
    const void* const* sets[1] = {cores};
    hipError_t e = prepare_tt<double>(p, sets, nullptr, ws, stream, "quality_tt_f64", a);
    if (e != hipSuccess) return e;
    const int64_t tiles = p.n_mid * ((p.NL + 16 * kQualNpb - 1) / (16 * kQualNpb));
    const size_t lds = quality_lds(p.n_last);
    KernelTimer tk("quality_tt_f64", stream);
#define LRC_TQ(K) \
    hipLaunchKernelGGL((k_tt_wave_q<K>), dim3((unsigned)G), dim3(256), lds, stream, a, tiles, X, scale, part, part2)
    switch (p.wave_nkb) {
    case 4: LRC_TQ(4); break;
    case 5: LRC_TQ(5); break;
    case 8: LRC_TQ(8); break;
    case 9: LRC_TQ(9); break;
    case 12: LRC_TQ(12); break;
    case 16: LRC_TQ(16); break;
    case 17: LRC_TQ(17); break;
    default: return hipErrorInvalidValue;
    }
#undef LRC_TQ
    return hipGetLastError();
}

}  // namespace lrc

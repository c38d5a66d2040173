// Fused Tensor-Train reconstruction for gfx950 (Sec. 5.1; Sec. 7.5
// eq. gpu_tt_reconstruction).
//
// The paper contracts the cores left to right, B_l = Z_{l-1} K_l, through
// preallocated buffers in global memory.  Here the dense tensor, viewed as a
// matrix with rows (i_1..i_{d-1}) and columns i_d, is cut into blocks of
// P rows; one workgroup produces a block entirely on chip:
//   1. left interface rows Z_{d-2}(L) for BL consecutive left indices
//      L = (i_1..i_{d-2}), computed level by level in LDS (VALU, the
//      accumulation precision) -- for d = 3 these are rows of G_1;
//   2. the middle contraction Z_{d-1}(L, i) = Z_{d-2}(L) G_{d-1}(i) for BI
//      middle indices i, on the matrix cores, into LDS;
//   3. the last contraction out(L, i, :) = Z_{d-1}(L, i) G_d, on the matrix
//      cores, stored straight from the accumulators (four consecutive
//      outputs per lane for FP32/FP16).
// Only the cores are read and only the tensor is written: no interface
// matrix goes to HBM.  For FP16 the accumulation is FP32 and the interface
// Z_{d-1} is rounded once to FP16 as the input of the last product; the
// FP16 middle and last cores are first copied to K-contiguous, zero-padded
// layouts (a few KB to MB) so each lane loads its 8 K values at once.
#include <algorithm>

#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

struct TTArgs {
    const void* core[kMaxD];
    int64_t dims[kMaxD];
    int64_t ranks[kMaxD + 1];
    int64_t divs[kMaxD];     // divs[c] = prod of dims[c+1 .. d-3] (left chain)
    int d;
    int64_t NL, n_mid, n_last;
    int rL, rM, Kp2, Kp3, Rt;
    int BL, BI, P, BLpad;
    int zf_off, cb_off;      // byte offsets of Z_{d-1} and the chain buffers in LDS
    int64_t num_L_blocks;
    int chain_rmax;
    const void* st_mid;      // FP16 only: [n_mid][Rt][Kp2]
    const void* st_last;     // FP16 only: [n_last][Kp3]
    void* out;
    int vec4;
};

// Copies of the FP16 middle and last cores with the contraction index
// contiguous and zero padding (tiny; done once per call).
__global__ __launch_bounds__(256) void k_stage_f16(const half_t* __restrict__ gmid, const half_t* __restrict__ glast,
                                                   half_t* __restrict__ smid, half_t* __restrict__ slast,
                                                   int64_t n_mid, int64_t n_last, int rL, int rM, int Kp2, int Kp3,
                                                   int Rt) {
    const int64_t tot_mid = n_mid * Rt * Kp2;
    const int64_t tot_last = n_last * Kp3;
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < tot_mid + tot_last; idx += stride) {
        if (idx < tot_mid) {
            const int64_t s = idx % Kp2, t = (idx / Kp2) % Rt, i = idx / ((int64_t)Kp2 * Rt);
            smid[idx] = (t < rM && s < rL) ? gmid[(s * n_mid + i) * rM + t] : half_t(0);
        } else {
            const int64_t j = idx - tot_mid;
            const int64_t t = j % Kp3, c = j / Kp3;
            slast[j] = (t < rM) ? glast[t * n_last + c] : half_t(0);
        }
    }
}

// A-operand fragment of the middle product: rows t, K index s, middle index i.
template <typename T>
__device__ __forceinline__ typename PrecTraits<T>::frag mid_frag(const TTArgs& a, int64_t i, int t, int s0);
template <>
__device__ __forceinline__ double mid_frag<double>(const TTArgs& a, int64_t i, int t, int s0) {
    const double* g = static_cast<const double*>(a.core[a.d - 2]);
    return (t < a.rM && s0 < a.rL && i < a.n_mid) ? g[((int64_t)s0 * a.n_mid + i) * a.rM + t] : 0.0;
}
template <>
__device__ __forceinline__ float mid_frag<float>(const TTArgs& a, int64_t i, int t, int s0) {
    const float* g = static_cast<const float*>(a.core[a.d - 2]);
    return (t < a.rM && s0 < a.rL && i < a.n_mid) ? g[((int64_t)s0 * a.n_mid + i) * a.rM + t] : 0.0f;
}
template <>
__device__ __forceinline__ half8_t mid_frag<half_t>(const TTArgs& a, int64_t i, int t, int s0) {
    if (i >= a.n_mid) {
        half8_t z;
#pragma unroll
        for (int e = 0; e < 8; ++e) z[e] = 0;
        return z;
    }
    const half_t* st = static_cast<const half_t*>(a.st_mid);
    return *reinterpret_cast<const half8_t*>(st + (i * a.Rt + t) * a.Kp2 + s0);
}

// A-operand fragment of the last product: rows c, K index t.
template <typename T>
__device__ __forceinline__ typename PrecTraits<T>::frag last_frag(const TTArgs& a, int64_t c, int t0);
template <>
__device__ __forceinline__ double last_frag<double>(const TTArgs& a, int64_t c, int t0) {
    const double* g = static_cast<const double*>(a.core[a.d - 1]);
    return (t0 < a.rM && c < a.n_last) ? g[(int64_t)t0 * a.n_last + c] : 0.0;
}
template <>
__device__ __forceinline__ float last_frag<float>(const TTArgs& a, int64_t c, int t0) {
    const float* g = static_cast<const float*>(a.core[a.d - 1]);
    return (t0 < a.rM && c < a.n_last) ? g[(int64_t)t0 * a.n_last + c] : 0.0f;
}
template <>
__device__ __forceinline__ half8_t last_frag<half_t>(const TTArgs& a, int64_t c, int t0) {
    if (c >= a.n_last) {
        half8_t z;
#pragma unroll
        for (int e = 0; e < 8; ++e) z[e] = 0;
        return z;
    }
    const half_t* st = static_cast<const half_t*>(a.st_last);
    return *reinterpret_cast<const half8_t*>(st + c * a.Kp3 + t0);
}

// Left interface rows Z_{d-2}(L) for L in [L0, L0 + BL) into Zl[BLpad][Kp2]
// (storage type; rows >= BL and columns >= rL are zero).
template <typename T>
__device__ void build_left(const TTArgs& a, int64_t L0, T* Zl, typename PrecTraits<T>::acc* cb0,
                           typename PrecTraits<T>::acc* cb1) {
    using Acc = typename PrecTraits<T>::acc;
    const int tid = threadIdx.x;
    const int total = a.BLpad * a.Kp2;
    if (a.d == 2) {
        for (int idx = tid; idx < total; idx += 256) Zl[idx] = (idx == 0) ? T(1) : T(0);
        return;
    }
    if (a.d == 3) {
        const T* g1 = static_cast<const T*>(a.core[0]);
        for (int idx = tid; idx < total; idx += 256) {
            const int Lr = idx / a.Kp2, s = idx % a.Kp2;
            const int64_t L = L0 + Lr;
            Zl[idx] = (Lr < a.BL && L < a.NL && s < a.rL) ? g1[L * a.rL + s] : T(0);
        }
        return;
    }
    // d >= 4: levels c = 0 .. d-3 (cores of the left chain)
    const int64_t Lend = (L0 + a.BL < a.NL) ? L0 + a.BL : a.NL;
    Acc* cur = cb0;
    Acc* nxt = cb1;
    int64_t qlo_prev = 0;
    for (int c = 0; c <= a.d - 3; ++c) {
        const int64_t D = a.divs[c];
        const int64_t qlo = L0 / D, qhi = (Lend - 1) / D;
        const int cnt = (int)(qhi - qlo + 1);
        const int r1 = (int)a.ranks[c + 1];
        const int64_t nc = a.dims[c];
        const T* g = static_cast<const T*>(a.core[c]);
        if (c == 0) {
            for (int idx = tid; idx < cnt * r1; idx += 256) {
                const int ql = idx / r1, t = idx % r1;
                nxt[ql * a.chain_rmax + t] = to_acc(g[(qlo + ql) * r1 + t]);
            }
        } else {
            const int r0 = (int)a.ranks[c];
            for (int idx = tid; idx < cnt * r1; idx += 256) {
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
    // cur holds Z_{d-2} rows for L in [L0, Lend) (divs[d-3] = 1)
    for (int idx = tid; idx < total; idx += 256) {
        const int Lr = idx / a.Kp2, s = idx % a.Kp2;
        const bool ok = (Lr < a.BL) && (L0 + Lr < a.NL) && (s < a.rL);
        Zl[idx] = ok ? to_storage<T>(cur[Lr * a.chain_rmax + s]) : T(0);
    }
}

template <typename T>
__global__ __launch_bounds__(256) void k_tt_fused(TTArgs a) {
    using Acc = typename PrecTraits<T>::acc;
    using AccV = typename PrecTraits<T>::accv;
    using Frag = typename PrecTraits<T>::frag;
    constexpr int KB = PrecTraits<T>::KB, KPL = PrecTraits<T>::KPL;
    extern __shared__ double4_t smem_v[];
    char* smem = reinterpret_cast<char*>(smem_v);
    T* Zl = reinterpret_cast<T*>(smem);
    T* Zf = reinterpret_cast<T*>(smem + a.zf_off);
    Acc* cb0 = reinterpret_cast<Acc*>(smem + a.cb_off);
    Acc* cb1 = cb0 + (size_t)a.BL * a.chain_rmax;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int64_t i0 = (int64_t)blockIdx.x * a.BI;

    // Z_{d-1} columns [min(Rt, Kp3), Kp3) are never written by the middle
    // product; clear the whole buffer once.
    for (int idx = tid; idx < a.P * a.Kp3; idx += 256) Zf[idx] = T(0);

    const int n_tb = a.Rt / 16;
    const int n_Lb = a.BLpad / 16;
    const int n_kb2 = a.Kp2 / KB;
    const int n_kb3 = a.Kp3 / KB;
    const int n_pb = a.P / 16;
    const int n_cb = (int)((a.n_last + 15) / 16);
    const int tcap = (a.Rt < a.Kp3) ? a.Rt : a.Kp3;

    for (int64_t lb = blockIdx.y; lb < a.num_L_blocks; lb += gridDim.y) {
        const int64_t L0 = lb * a.BL;
        __syncthreads();   // previous block's readers of Zl / Zf are done
        build_left<T>(a, L0, Zl, cb0, cb1);
        __syncthreads();

        // middle product: items (il, tb, Lb)
        const int n_items = a.BI * n_tb * n_Lb;
        for (int it = wave; it < n_items; it += 4) {
            const int il = it / (n_tb * n_Lb);
            const int tb = (it / n_Lb) % n_tb;
            const int Lb = it % n_Lb;
            AccV acc = zero_accv<AccV>();
            for (int kb = 0; kb < n_kb2; ++kb) {
                const int s0 = kb * KB + g * KPL;
                const Frag fa = mid_frag<T>(a, i0 + il, tb * 16 + r, s0);
                const Frag fb = load_frag<T>(Zl + (Lb * 16 + r) * a.Kp2 + s0);
                acc = mfma(fa, fb, acc);
            }
            const int Lr = Lb * 16 + r;
            if (Lr < a.BL) {
                T* dst = Zf + (Lr * a.BI + il) * a.Kp3;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int t = tb * 16 + acc_row<T>(g, v);
                    if (t < tcap) dst[t] = to_storage<T>(acc[v]);
                }
            }
        }
        __syncthreads();

        // last product and stores
        for (int cbk = wave; cbk < n_cb; cbk += 4) {
            const int64_t c = (int64_t)cbk * 16 + r;
            AccV acc[4];
#pragma unroll
            for (int pb = 0; pb < 4; ++pb) acc[pb] = zero_accv<AccV>();
            for (int kb = 0; kb < n_kb3; ++kb) {
                const int t0 = kb * KB + g * KPL;
                const Frag fa = last_frag<T>(a, c, t0);
#pragma unroll
                for (int pb = 0; pb < 4; ++pb) {
                    if (pb < n_pb) {
                        const Frag fb = load_frag<T>(Zf + (pb * 16 + r) * a.Kp3 + t0);
                        acc[pb] = mfma(fa, fb, acc[pb]);
                    }
                }
            }
            const int64_t cb0 = (int64_t)cbk * 16;
#pragma unroll
            for (int pb = 0; pb < 4; ++pb) {
                if (pb >= n_pb) continue;
                const int p = pb * 16 + r;
                const int Lr = p / a.BI, il = p % a.BI;
                const int64_t L = L0 + Lr, i = i0 + il;
                if (Lr >= a.BL || L >= a.NL || i >= a.n_mid) continue;
                T* dst = static_cast<T*>(a.out) + (L * a.n_mid + i) * a.n_last + cb0;
                if (AccRowsContiguous<T>::value && a.vec4 && cb0 + 4 * g + 3 < a.n_last) {
                    typedef T vec_t __attribute__((ext_vector_type(4)));
                    vec_t w;
#pragma unroll
                    for (int v = 0; v < 4; ++v) w[v] = to_storage<T>(acc[pb][v]);
                    *reinterpret_cast<vec_t*>(dst + 4 * g) = w;
                } else {
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const int row = acc_row<T>(g, v);
                        if (cb0 + row < a.n_last) dst[row] = to_storage<T>(acc[pb][v]);
                    }
                }
            }
        }
    }
}

int plan_tt(TTPlan& p, const int64_t* dims, const int64_t* ranks, int d, int prec, size_t max_lds) {
    p = TTPlan{};
    p.d = d;
    p.prec = prec;
    for (int c = 0; c < d; ++c) p.dims[c] = dims[c];
    for (int c = 0; c <= d; ++c) p.ranks[c] = ranks[c];
    const int KB = mfma_kb(prec);
    const int e = elem_bytes(prec);
    const int acc_b = (prec == P64) ? 8 : 4;
    p.n_last = dims[d - 1];
    p.n_mid = dims[d - 2];
    p.rM = (int)ranks[d - 1];
    p.rL = (int)ranks[d - 2];
    p.NL = 1;
    for (int c = 0; c <= d - 3; ++c) p.NL *= dims[c];
    p.Kp2 = (int)round_up(p.rL, KB);
    p.Kp3 = (int)round_up(p.rM, KB);
    p.Rt = (int)round_up(p.rM, 16);
    p.chain_rmax = 1;
    if (d >= 4)
        for (int c = 1; c <= d - 2; ++c) p.chain_rmax = (int)std::max<int64_t>(p.chain_rmax, ranks[c]);
    const int P0 = (prec == P64) ? 32 : 64;
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
        size_t lds = (size_t)round_up((int64_t)BLpad * p.Kp2 * e, 32) + (size_t)round_up((int64_t)Peff * p.Kp3 * e, 32);
        if (d >= 4) lds += (size_t)2 * BL * p.chain_rmax * acc_b;
        if (Peff > 64) continue;
        if (lds <= max_lds) {
            p.BL = BL;
            p.BI = BI;
            p.P = Peff;
            p.lds_bytes = lds;
            break;
        }
    }
    if (p.P == 0) return -1;
    p.num_i_blocks = (p.n_mid + p.BI - 1) / p.BI;
    p.num_L_blocks = (p.NL + p.BL - 1) / p.BL;
    int64_t want = 4096 / std::max<int64_t>(1, p.num_i_blocks);
    if (want < 1) want = 1;
    if (want > p.num_L_blocks) want = p.num_L_blocks;
    if (want > 65535) want = 65535;
    p.grid_L = (int)want;
    p.stage_bytes = (prec == P16) ? (size_t)(round_up(p.n_mid * p.Rt * p.Kp2 * 2, 256) + round_up(p.n_last * p.Kp3 * 2, 256)) : 0;
    return 0;
}

template <typename T>
static hipError_t tt_typed(const TTPlan& p, const void* const* cores, void* out, Workspace& ws,
                           hipStream_t stream, const char* label) {
    TTArgs a{};
    a.d = p.d;
    for (int c = 0; c < p.d; ++c) {
        a.core[c] = cores[c];
        a.dims[c] = p.dims[c];
    }
    for (int c = 0; c <= p.d; ++c) a.ranks[c] = p.ranks[c];
    for (int c = 0; c <= p.d - 3; ++c) {
        int64_t D = 1;
        for (int c2 = c + 1; c2 <= p.d - 3; ++c2) D *= p.dims[c2];
        a.divs[c] = D;
    }
    a.NL = p.NL;
    a.n_mid = p.n_mid;
    a.n_last = p.n_last;
    a.rL = p.rL;
    a.rM = p.rM;
    a.Kp2 = p.Kp2;
    a.Kp3 = p.Kp3;
    a.Rt = p.Rt;
    a.BL = p.BL;
    a.BI = p.BI;
    a.P = p.P;
    a.BLpad = (int)round_up(p.BL, 16);
    a.zf_off = (int)round_up((int64_t)a.BLpad * p.Kp2 * (int64_t)sizeof(T), 32);
    a.cb_off = a.zf_off + (int)round_up((int64_t)p.P * p.Kp3 * (int64_t)sizeof(T), 32);
    a.num_L_blocks = p.num_L_blocks;
    a.chain_rmax = p.chain_rmax;
    a.out = out;
    a.vec4 = (p.n_last % 4 == 0) && (reinterpret_cast<uintptr_t>(out) % (4 * sizeof(T)) == 0);
    if (p.prec == P16) {
        half_t* smid = static_cast<half_t*>(ws.take((size_t)p.n_mid * p.Rt * p.Kp2 * 2));
        half_t* slast = static_cast<half_t*>(ws.take((size_t)p.n_last * p.Kp3 * 2));
        if (ws.overrun || !smid || !slast) return hipErrorOutOfMemory;
        const int64_t tot = p.n_mid * p.Rt * p.Kp2 + p.n_last * p.Kp3;
        int64_t gs = (tot + 255) / 256;
        if (gs > 2048) gs = 2048;
        KernelTimer ts("tt_stage_f16", stream);
        hipLaunchKernelGGL(k_stage_f16, dim3((unsigned)gs), dim3(256), 0, stream, (const half_t*)cores[p.d - 2],
                           (const half_t*)cores[p.d - 1], smid, slast, p.n_mid, p.n_last, p.rL, p.rM, p.Kp2, p.Kp3,
                           p.Rt);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        a.st_mid = smid;
        a.st_last = slast;
    }
    dim3 grid((unsigned)p.num_i_blocks, (unsigned)p.grid_L);
    if (!label) label = p.prec == P64 ? "tt_fused_f64" : (p.prec == P32 ? "tt_fused_f32" : "tt_fused_f16");
    KernelTimer tk(label, stream);
    hipLaunchKernelGGL(k_tt_fused<T>, grid, dim3(256), p.lds_bytes, stream, a);
    return hipGetLastError();
}

hipError_t launch_tt(const TTPlan& p, const void* const* cores, void* out, Workspace& ws, hipStream_t stream,
                     const char* label) {
    if (p.prec == P64) return tt_typed<double>(p, cores, out, ws, stream, label);
    if (p.prec == P32) return tt_typed<float>(p, cores, out, ws, stream, label);
    return tt_typed<half_t>(p, cores, out, ws, stream, label);
}

}  // namespace lrc

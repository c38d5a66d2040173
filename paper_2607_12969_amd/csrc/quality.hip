// Quality of a reconstruction against its FP64 reference, for the
// fixed-memory comparison (Sec. sec:hyperspectral_application): relative
// Frobenius error, band-wise PSNR, the SSIM variant evaluated once per whole
// band, and the spectral angle mapper.  The spectral bands are the last
// (contiguous) mode, the pixels all leading indices: X and Xh are P x B
// row-major, Xh scaled by `scale` (undoing a normalization) as it is read.
//
// Two passes over the pair, each HBM-bound (16 bytes per FP64 entry pair):
//   k_band_stats  per workgroup of pixel rows and per band, shifted sums
//                 (shift s_b = X[0][b], against cancellation in the
//                 variances), the squared differences and squares, and the
//                 band's minimum and maximum;
//   k_sam         one wave per pixel: dot product and squared norms over the
//                 bands, the angle, summed per workgroup.
// k_quality_reduce adds the row blocks' partials (one wave per statistic
// and band) and k_quality_finish forms the per-band measures and their
// means, both in a fixed order (bitwise reproducible results).
#include <hip/hip_runtime.h>

#include "lrc_device.h"
#include "lrc_internal.h"

namespace lrc {

template <typename Y>
__device__ __forceinline__ double widen_q(Y v) { return static_cast<double>(v); }

// part[(blk * QS_N + q) * B + b]
template <typename Y>
__global__ __launch_bounds__(256) void k_band_stats(const double* __restrict__ X, const Y* __restrict__ Xh,
                                                    double scale, int64_t P, int64_t B, int64_t rows_per_blk,
                                                    double* __restrict__ part) {
    const int64_t p0 = (int64_t)blockIdx.x * rows_per_blk;
    const int64_t p1 = p0 + rows_per_blk < P ? p0 + rows_per_blk : P;
    for (int64_t b = threadIdx.x; b < B; b += 256) {
        const double s = X[b];
        double sx = 0, sy = 0, sxx = 0, syy = 0, sxy = 0, sdd = 0, s2 = 0;
        double mn = s, mx = s;
        int64_t p = p0;
        // four rows per step: their loads are in flight together
        for (; p + 3 < p1; p += 4) {
            double x[4], y[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                x[u] = X[(p + u) * B + b];
                y[u] = scale * widen_q(Xh[(p + u) * B + b]);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const double dx = x[u] - s, dy = y[u] - s, dd = x[u] - y[u];
                sx += dx;
                sy += dy;
                sxx += dx * dx;
                syy += dy * dy;
                sxy += dx * dy;
                sdd += dd * dd;
                s2 += x[u] * x[u];
                mn = x[u] < mn ? x[u] : mn;
                mx = x[u] > mx ? x[u] : mx;
            }
        }
        for (; p < p1; ++p) {
            const double x = X[p * B + b], y = scale * widen_q(Xh[p * B + b]);
            const double dx = x - s, dy = y - s, dd = x - y;
            sx += dx;
            sy += dy;
            sxx += dx * dx;
            syy += dy * dy;
            sxy += dx * dy;
            sdd += dd * dd;
            s2 += x * x;
            mn = x < mn ? x : mn;
            mx = x > mx ? x : mx;
        }
        double* o = part + (int64_t)blockIdx.x * QS_N * B + b;
        o[QS_X * B] = sx;
        o[QS_Y * B] = sy;
        o[QS_XX * B] = sxx;
        o[QS_YY * B] = syy;
        o[QS_XY * B] = sxy;
        o[QS_DD * B] = sdd;
        o[QS_X2 * B] = s2;
        o[QS_MIN * B] = mn;
        o[QS_MAX * B] = mx;
    }
}

// part2[2 blk] = sum of angles, part2[2 blk + 1] = pixels counted
template <typename Y>
__global__ __launch_bounds__(256) void k_sam(const double* __restrict__ X, const Y* __restrict__ Xh, double scale,
                                             int64_t P, int64_t B, double* __restrict__ part2) {
    __shared__ double ws[4][2];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    double asum = 0.0, cnt = 0.0;
    for (int64_t p = (int64_t)blockIdx.x * 4 + wave; p < P; p += (int64_t)gridDim.x * 4) {
        double dot = 0.0, xx = 0.0, yy = 0.0;
        for (int64_t b = lane; b < B; b += 64) {
            const double x = X[p * B + b], y = scale * widen_q(Xh[p * B + b]);
            dot += x * y;
            xx += x * x;
            yy += y * y;
        }
        dot = wave_sum(dot);
        xx = wave_sum(xx);
        yy = wave_sum(yy);
        const double nn = __builtin_sqrt(xx) * __builtin_sqrt(yy);
        if (nn > 0.0) {
            double c = dot / nn;
            c = c > 1.0 ? 1.0 : (c < -1.0 ? -1.0 : c);
            asum += acos(c);
            cnt += 1.0;
        }
    }
    if (lane == 0) {
        ws[wave][0] = asum;
        ws[wave][1] = cnt;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double a = 0.0, c = 0.0;
        for (int w = 0; w < 4; ++w) {
            a += ws[w][0];
            c += ws[w][1];
        }
        part2[2 * blockIdx.x] = a;
        part2[2 * blockIdx.x + 1] = c;
    }
}

// red[q * B + b] = the band sums (minimum / maximum for QS_MIN / QS_MAX)
// over the nblk row blocks: one wave per (q, b), lane j taking blocks
// j, j + 64, ... in order, then a fixed butterfly.
__global__ __launch_bounds__(256) void k_quality_reduce(const double* __restrict__ part, int64_t nblk, int64_t B,
                                                        double* __restrict__ red) {
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (w >= QS_N * B) return;
    const int q = (int)(w / B);
    const int64_t b = w - (int64_t)q * B;
    const double* src = part + (int64_t)q * B + b;
    const int64_t stride = (int64_t)QS_N * B;
    const bool mn = q == QS_MIN, mxq = q == QS_MAX;
    double v = (mn || mxq) ? src[0] : 0.0;
    for (int64_t k = lane; k < nblk; k += 64) {
        const double o = src[k * stride];
        v = mn ? (o < v ? o : v) : (mxq ? (o > v ? o : v) : v + o);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const double o = __shfl_xor(v, off, 64);
        v = mn ? (o < v ? o : v) : (mxq ? (o > v ? o : v) : v + o);
    }
    if (lane == 0) red[w] = v;
}

// out: rel_err, mean PSNR, mean SSIM, mean SAM, SAM pixel count (red: the
// band sums of k_quality_reduce)
__global__ __launch_bounds__(256) void k_quality_finish(const double* __restrict__ red,
                                                        const double* __restrict__ part2, int64_t nblk2,
                                                        const double* __restrict__ X, int64_t P, int64_t B,
                                                        double* __restrict__ out) {
    __shared__ double acc[256][6];   // per thread: PSNR_b, SSIM_b, squared differences, squares, angles, pixels
    const int t = threadIdx.x;
    double ps = 0.0, ss = 0.0, dd = 0.0, x2 = 0.0, sa = 0.0, sc = 0.0;
    // the angle partials: thread t adds blocks t, t + 256, ... in order
    for (int64_t k = t; k < nblk2; k += 256) {
        sa += part2[2 * k];
        sc += part2[2 * k + 1];
    }
    const double np = (double)P;
    for (int64_t b = t; b < B; b += 256) {
        double v[QS_N];
        for (int q = 0; q < QS_N; ++q) v[q] = red[q * B + b];
        // L_b: range of the reference band, max(max|X_b|, 1) when constant
        double L = v[QS_MAX] - v[QS_MIN];
        if (!(L > 0.0)) {
            const double a = fabs(v[QS_MIN]) > fabs(v[QS_MAX]) ? fabs(v[QS_MIN]) : fabs(v[QS_MAX]);
            L = a > 1.0 ? a : 1.0;
        }
        const double mse = v[QS_DD] / np;
        ps += 20.0 * log10(L / sqrt(mse));   // +inf for an exact band
        const double s = X[b];
        const double ex = v[QS_X] / np, ey = v[QS_Y] / np;   // shifted means
        const double mx = s + ex, my = s + ey;
        const double vx = v[QS_XX] / np - ex * ex, vy = v[QS_YY] / np - ey * ey;
        const double cxy = v[QS_XY] / np - ex * ey;
        const double c1 = (0.01 * L) * (0.01 * L), c2 = (0.03 * L) * (0.03 * L);
        ss += (2.0 * mx * my + c1) * (2.0 * cxy + c2) / ((mx * mx + my * my + c1) * (vx + vy + c2));
        dd += v[QS_DD];
        x2 += v[QS_X2];
    }
    acc[t][0] = ps;
    acc[t][1] = ss;
    acc[t][2] = dd;
    acc[t][3] = x2;
    acc[t][4] = sa;
    acc[t][5] = sc;
    __syncthreads();
    if (t >= 64) return;
    // wave 0: lane l adds threads l, l + 64, l + 128, l + 192, then a fixed butterfly
    double a[6];
#pragma unroll
    for (int j = 0; j < 6; ++j) a[j] = wave_sum(((acc[t][j] + acc[t + 64][j]) + acc[t + 128][j]) + acc[t + 192][j]);
    if (t == 0) {
        const double a0 = a[0], a1 = a[1], a2 = a[2], a3 = a[3];
        sa = a[4];
        sc = a[5];
        out[0] = sqrt(a2) / sqrt(a3);
        out[1] = a0 / (double)B;
        out[2] = a1 / (double)B;
        out[3] = sc > 0.0 ? sa / sc : __builtin_nan("");
        out[4] = sc;
    }
}

static void quality_grid(int64_t P, int64_t* nblk, int64_t* rows, int64_t* nblk2) {
    // about 1024 row blocks of at least 64 rows for the band sums; 1024
    // workgroups (4 pixels at a time) for the angles
    int64_t r = (P + 1023) / 1024;
    if (r < 64) r = 64;
    *rows = r;
    *nblk = (P + r - 1) / r;
    int64_t g = (P + 3) / 4;
    *nblk2 = g < 1024 ? g : 1024;
}

size_t quality_workspace_bytes(int64_t P, int64_t B) {
    int64_t nblk, rows, nblk2;
    quality_grid(P, &nblk, &rows, &nblk2);
    return round_up(nblk * QS_N * B * 8, 256) + round_up(QS_N * B * 8, 256) + round_up(nblk2 * 2 * 8, 256) + 256;
}

template <typename Y>
static hipError_t quality_typed(const double* X, const Y* Xh, double scale, int64_t P, int64_t B, double* out,
                                Workspace& ws, hipStream_t stream) {
    int64_t nblk, rows, nblk2;
    quality_grid(P, &nblk, &rows, &nblk2);
    double* part = static_cast<double*>(ws.take((size_t)(nblk * QS_N * B * 8)));
    double* red = static_cast<double*>(ws.take((size_t)(QS_N * B * 8)));
    double* part2 = static_cast<double*>(ws.take((size_t)(nblk2 * 2 * 8)));
    if (ws.overrun) return hipErrorOutOfMemory;
    KernelTimer t("quality_f64", stream);
    hipLaunchKernelGGL((k_band_stats<Y>), dim3((unsigned)nblk), dim3(256), 0, stream, X, Xh, scale, P, B, rows,
                       part);
    hipLaunchKernelGGL((k_sam<Y>), dim3((unsigned)nblk2), dim3(256), 0, stream, X, Xh, scale, P, B, part2);
    hipLaunchKernelGGL(k_quality_reduce, dim3((unsigned)((QS_N * B + 3) / 4)), dim3(256), 0, stream, part, nblk, B,
                       red);
    hipLaunchKernelGGL(k_quality_finish, dim3(1), dim3(256), 0, stream, red, part2, nblk2, X, P, B, out);
    return hipGetLastError();
}

hipError_t launch_quality_reduce(const double* part, int64_t nblk, const double* part2, int64_t nblk2,
                                 const double* X, int64_t P, int64_t B, double* red, double* out,
                                 hipStream_t stream) {
    KernelTimer t("quality_f64", stream);
    hipLaunchKernelGGL(k_quality_reduce, dim3((unsigned)((QS_N * B + 3) / 4)), dim3(256), 0, stream, part, nblk, B,
                       red);
    hipLaunchKernelGGL(k_quality_finish, dim3(1), dim3(256), 0, stream, red, part2, nblk2, X, P, B, out);
    return hipGetLastError();
}

hipError_t launch_quality(const double* X, const void* Xh, int prec, double scale, int64_t P, int64_t B,
                          double* out, Workspace& ws, hipStream_t stream) {
    if (prec == P64) return quality_typed(X, static_cast<const double*>(Xh), scale, P, B, out, ws, stream);
    if (prec == P32) return quality_typed(X, static_cast<const float*>(Xh), scale, P, B, out, ws, stream);
    return quality_typed(X, static_cast<const half_t*>(Xh), scale, P, B, out, ws, stream);
}

}  // namespace lrc

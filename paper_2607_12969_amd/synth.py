"""Seeded synthetic inputs for the rank-compensation hot path.

This module only *draws* input data, in float64: Haar-distributed orthogonal
factors, prescribed singular-value laws, Gaussian batches, tensors defined by
a closed formula, and Tensor-Train generator cores with prescribed spectra.
It performs none of the method's own arithmetic: no truncation, no rounding
to FP32/FP16, no factor apply, no core contraction and no certificate.  Both
the GPU path and the CPU oracle consume what it returns.

Seeds: every stream is ``numpy.random.default_rng([12969, workload_id,
stream_id])`` (PCG64).  Stream ids: 0 = left factor, 1 = right factor,
2 = spectrum noise, 3 = batch X, 4 and up = tensor cores, endmembers,
abundances and noise; 10 and 11 = the full orthogonal factors of the dense
8192 x 8192 matrix.

Workloads stand in for the paper's data sets, which are not available here:
the matrix workloads replace the SuiteSparse application timings (Sec. 4.4)
and the tensor workloads replace the synthetic and public TT tests
(Sec. 7.2-7.5); shapes follow the paper's timing ranks (r 40->41 style +1
compensation, TT 32->36 and 64->65 schedules).
"""
from __future__ import annotations

import math

import numpy as np

SEED = 12969

# Workload ids (the first entry of every seed sequence).
W_MATRIX_SMALL = 1        # 512 x 256, sigma_j = 10^(-4(j-1)/255)
W_MATRIX_SQUARE = 2       # 8192 x 8192, sigma_j = j^-1.5 + 1e-8 noise
W_MATRIX_TAIL = 3         # 65536 x 4096, sigma_j = max(exp(-j/40), 1e-6)
W_TT_CUBE = 4             # 256^3 from rank-(24,24) generator cores
W_TT_SIXWAY = 5           # 16^6 from rank-(8,16,24,16,8) generator cores
W_TT_HYPER = 6            # 512 x 512 x 224 hyperspectral-shaped cube
W_RANDOM = 7              # generic shapes for kernel tests


def rng_for(workload: int, stream: int, extra: int = 0) -> np.random.Generator:
    return np.random.default_rng([SEED, int(workload), int(stream), int(extra)])


def haar(rng: np.random.Generator, m: int, n: int) -> np.ndarray:
    """m x n matrix with orthonormal columns, Haar distributed (the first n
    columns of a Haar orthogonal matrix): QR of a Gaussian with the signs of
    diag(R) moved into Q (Mezzadri's construction)."""
    if n > m:
        raise ValueError("haar: need n <= m")
    g = rng.standard_normal((m, n))
    q, r = np.linalg.qr(g)
    d = np.sign(np.diag(r))
    d[d == 0] = 1.0
    return np.ascontiguousarray(q * d)


def gaussian(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(shape)


# --------------------------------------------------------------------------
# Matrix workloads
# --------------------------------------------------------------------------

def matrix_small():
    """512 x 256 matrix A = Q1[:, :256] diag(sigma) Q2^T with
    sigma_j = 10^(-4(j-1)/255), Haar Q1 (512 x 512) and Q2 (256 x 256),
    and a 256 x 64 standard-normal batch.  Dense A is cheap here, so it is
    returned too.  Base rank 20 (FP64), compensated rank 21."""
    m, n = 512, 256
    j = np.arange(1, n + 1, dtype=np.float64)
    sigma = 10.0 ** (-4.0 * (j - 1.0) / 255.0)
    q1 = haar(rng_for(W_MATRIX_SMALL, 0), m, m)[:, :n]
    q2 = haar(rng_for(W_MATRIX_SMALL, 1), n, n)
    a = (q1 * sigma) @ q2.T
    x = gaussian(rng_for(W_MATRIX_SMALL, 3), (n, 64))
    return dict(m=m, n=n, A=a, sigma=sigma, U=q1, V=q2, X=x, k=20)


def sigma_square(n: int = 8192) -> np.ndarray:
    """Algebraic decay j^-1.5 with additive Gaussian noise at 1e-8 * sigma_1
    on the spectrum, absolute value, sorted non-increasing."""
    j = np.arange(1, n + 1, dtype=np.float64)
    g = rng_for(W_MATRIX_SQUARE, 2).standard_normal(n)
    s = np.abs(j ** -1.5 + 1e-8 * g)
    return np.sort(s)[::-1].copy()


def sigma_tail(n: int = 4096) -> np.ndarray:
    """sigma_j = max(exp(-j/40), 1e-6), j = 1..n (already non-increasing)."""
    j = np.arange(1, n + 1, dtype=np.float64)
    return np.maximum(np.exp(-j / 40.0), 1e-6)


def matrix_square(kmax: int = 256, batch: int = 4096, m: int = 8192, n: int = 8192):
    """Leading kmax+1 singular triplets of an m x n matrix with Haar singular
    vectors and the sigma_square law, plus an n x batch Gaussian batch.
    The SVD is known by construction; the dense matrix is never formed."""
    r = kmax + 1
    u = haar(rng_for(W_MATRIX_SQUARE, 0), m, r)
    v = haar(rng_for(W_MATRIX_SQUARE, 1), n, r)
    sigma = sigma_square(min(m, n))
    x = gaussian(rng_for(W_MATRIX_SQUARE, 3), (n, batch))
    return dict(m=m, n=n, U=u, V=v, sigma=sigma, X=x)


def matrix_square_dense(kmax: int = 256, m: int = 8192, n: int = 8192):
    """The 8192 x 8192 workload formed densely, for the error of the stored
    representation against A itself: full Haar orthogonal Q1 (m x m) and
    Q2 (n x n) from streams 10 and 11, A = Q1 diag(sigma) Q2^T with the
    sigma_square law over all min(m, n) values.  Returns A with its leading
    kmax+1 singular triplets (the first columns of Q1 and Q2)."""
    r = kmax + 1
    sigma = sigma_square(min(m, n))
    q1 = haar(rng_for(W_MATRIX_SQUARE, 10), m, m)
    q2 = haar(rng_for(W_MATRIX_SQUARE, 11), n, n)
    a = (q1[:, :min(m, n)] * sigma) @ q2[:, :min(m, n)].T
    return dict(m=m, n=n, A=a, sigma=sigma, U=np.ascontiguousarray(q1[:, :r]), V=np.ascontiguousarray(q2[:, :r]))


def matrix_tail(kmax: int = 512, batch: int = 4096, m: int = 65536, n: int = 4096):
    """Leading kmax+1 singular triplets of the tail-rank stress matrix
    (sigma_tail law, Haar singular vectors) plus an n x batch batch."""
    r = kmax + 1
    u = haar(rng_for(W_MATRIX_TAIL, 0), m, r)
    v = haar(rng_for(W_MATRIX_TAIL, 1), n, r)
    sigma = sigma_tail(min(m, n))
    x = gaussian(rng_for(W_MATRIX_TAIL, 3), (n, batch))
    return dict(m=m, n=n, U=u, V=v, sigma=sigma, X=x)


def random_factors(m: int, n: int, r: int, batch: int, tag: int = 0):
    """Generic Haar factors with a geometric spectrum and a Gaussian batch,
    for kernel tests at arbitrary (ragged) shapes."""
    rr = max(1, min(r, m, n))
    u = np.zeros((m, r))
    v = np.zeros((n, r))
    u[:, :rr] = haar(rng_for(W_RANDOM, 0, tag), m, rr)
    v[:, :rr] = haar(rng_for(W_RANDOM, 1, tag), n, rr)
    if r > rr:  # more columns than the dimension allows: fill with Gaussians
        u[:, rr:] = rng_for(W_RANDOM, 5, tag).standard_normal((m, r - rr)) / math.sqrt(m)
        v[:, rr:] = rng_for(W_RANDOM, 6, tag).standard_normal((n, r - rr)) / math.sqrt(n)
    s = 0.9 ** np.arange(r, dtype=np.float64)
    x = gaussian(rng_for(W_RANDOM, 3, tag), (n, batch))
    return dict(U=u, s=s, V=v, X=x)


# --------------------------------------------------------------------------
# Tensors defined by formula (the paper's controlled synthetic tests)
# --------------------------------------------------------------------------

def hilbert_3d(n: int = 100) -> np.ndarray:
    """T(i,j,k) = 1/(i+j+k-2), 1-based indices (Sec. 7.2)."""
    i = np.arange(1, n + 1, dtype=np.float64)
    return 1.0 / (i[:, None, None] + i[None, :, None] + i[None, None, :] - 2.0)


def decay_3d(n: int = 60) -> np.ndarray:
    """T(i,j,k) = 1/(1+|i-j|+|j-k|+|i-k|) (Sec. 7.2)."""
    i = np.arange(1, n + 1, dtype=np.float64)
    a, b, c = i[:, None, None], i[None, :, None], i[None, None, :]
    return 1.0 / (1.0 + np.abs(a - b) + np.abs(b - c) + np.abs(a - c))


def _grid(n: int, d: int):
    i = np.arange(1, n + 1, dtype=np.float64)
    out = []
    for p in range(d):
        shape = [1] * d
        shape[p] = n
        out.append(i.reshape(shape))
    return out


def hilbert_6d(n: int = 12) -> np.ndarray:
    """T(i_1..i_6) = 1/(i_1+...+i_6-5) (Sec. 7.3)."""
    g = _grid(n, 6)
    s = sum(g)
    return 1.0 / (s - 5.0)


def decay_6d(n: int = 12) -> np.ndarray:
    """T = 1/(1 + sum_{p<q} |i_p - i_q|) (Sec. 7.3)."""
    g = _grid(n, 6)
    acc = 1.0
    for p in range(6):
        for q in range(p + 1, 6):
            acc = acc + np.abs(g[p] - g[q])
    return 1.0 / acc


# --------------------------------------------------------------------------
# Tensor-Train generator cores and the hyperspectral-shaped cube
# --------------------------------------------------------------------------

def _spectral_block(rng, rows: int, cols: int, spectrum: np.ndarray) -> np.ndarray:
    """rows x cols matrix Q diag(spectrum) W^T with Haar Q (rows x q) and
    Haar W (cols x q), q = len(spectrum) <= min(rows, cols)."""
    q = len(spectrum)
    left = haar(rng, rows, q)
    right = haar(rng, cols, q)
    return (left * spectrum) @ right.T


def tt_generator_cores(workload: int, dims, ranks, spectrum_fn, noise: float = 0.0):
    """Seeded generator cores G_l (r_{l-1} x n_l x r_l).  The left unfolding
    of every core but the last, and the right unfolding of the last core, is
    Q diag(|spectrum_j + noise * g_j|) W^T with Haar Q and W.  The tensor these
    cores define is the workload's input tensor (not normalised)."""
    d = len(dims)
    cores = []
    for l in range(d):
        rng = rng_for(workload, 4 + l)
        r0, n, r1 = int(ranks[l]), int(dims[l]), int(ranks[l + 1])
        if l < d - 1:
            q = min(r0 * n, r1)
            sp = np.abs(spectrum_fn(np.arange(q)) + noise * rng.standard_normal(q))
            mat = _spectral_block(rng, r0 * n, r1, sp)
            cores.append(np.ascontiguousarray(mat.reshape(r0, n, r1)))
        else:
            q = min(r0, n)
            sp = np.abs(spectrum_fn(np.arange(q)) + noise * rng.standard_normal(q))
            mat = _spectral_block(rng, r0, n, sp)
            cores.append(np.ascontiguousarray(mat.reshape(r0, n, 1)))
    return cores


def tt_cube_cores():
    """256^3 generator: ranks (1,24,24,1), spectra |2^-j + 1e-6 g_j|."""
    return tt_generator_cores(W_TT_CUBE, (256, 256, 256), (1, 24, 24, 1),
                              lambda j: 2.0 ** (-j.astype(np.float64)), noise=1e-6)


def tt_sixway_cores():
    """16^6 generator: ranks (1,8,16,24,16,8,1), spectra 1.5^-j."""
    return tt_generator_cores(W_TT_SIXWAY, (16,) * 6, (1, 8, 16, 24, 16, 8, 1),
                              lambda j: 1.5 ** (-j.astype(np.float64)), noise=0.0)


def _smooth_1d(x: np.ndarray, sigma: float, axis: int) -> np.ndarray:
    from scipy.ndimage import gaussian_filter1d
    return gaussian_filter1d(x, sigma, axis=axis, mode="reflect")


def hyperspectral(shape=(512, 512, 224), n_end: int = 8, noise: float = 1e-3) -> np.ndarray:
    """Hyperspectral-shaped cube standing in for the paper's public scenes
    (Sec. 7.4): n_end smooth nonnegative endmember spectra (white noise over
    the bands, Gaussian-smoothed with sigma = 8 bands, shifted to be >= 0)
    times abundance maps (Gaussian fields smoothed with sigma = 16 pixels,
    softmax across endmembers per pixel), plus noise at `noise` times the
    cube's rms, then scaled to unit Frobenius norm as the paper does for its
    public tensors."""
    h, w, b = shape
    rng_e = rng_for(W_TT_HYPER, 4)
    rng_a = rng_for(W_TT_HYPER, 5)
    rng_n = rng_for(W_TT_HYPER, 6)
    spec = _smooth_1d(rng_e.standard_normal((n_end, b)), 8.0, axis=1)
    spec = spec - spec.min(axis=1, keepdims=True)
    ab = rng_a.standard_normal((n_end, h, w))
    ab = _smooth_1d(_smooth_1d(ab, 16.0, axis=1), 16.0, axis=2)
    ab = ab / ab.std()
    ab = np.exp(ab - ab.max(axis=0, keepdims=True))
    ab = ab / ab.sum(axis=0, keepdims=True)
    t = ab.reshape(n_end, h * w).T @ spec            # (h*w) x b
    rms = math.sqrt(float(np.mean(t * t)))
    t += noise * rms * rng_n.standard_normal(t.shape)
    t /= np.linalg.norm(t)
    return t.reshape(h, w, b)


def random_tt_cores(dims, ranks, tag: int = 0):
    """Generic cores for kernel tests: left-orthogonal Haar cores for l < d
    (when r_l <= r_{l-1} n_l; Gaussian otherwise) and a last core whose rows
    decay geometrically, the shape TT-SVD output takes."""
    d = len(dims)
    cores = []
    for l in range(d):
        rng = rng_for(W_RANDOM, 8 + l, tag)
        r0, n, r1 = int(ranks[l]), int(dims[l]), int(ranks[l + 1])
        if l < d - 1:
            if r1 <= r0 * n:
                mat = haar(rng, r0 * n, r1)
            else:
                mat = rng.standard_normal((r0 * n, r1)) / math.sqrt(r0 * n)
            cores.append(np.ascontiguousarray(mat.reshape(r0, n, r1)))
        else:
            scale = 0.8 ** np.arange(r0, dtype=np.float64)
            mat = rng.standard_normal((r0, n)) * scale[:, None]
            cores.append(np.ascontiguousarray(mat.reshape(r0, n, 1)))
    return cores


# --------------------------------------------------------------------------
# Factorization inputs
# --------------------------------------------------------------------------

W_FACTOR = 8              # test vectors and dense matrices of the randomized factorizations


def test_vectors(l: int, n: int, tag: int = 0) -> np.ndarray:
    """l Gaussian test vectors of length n as the rows of an l x n matrix
    (the sketch of a randomized range finder)."""
    return rng_for(W_FACTOR, 0, tag).standard_normal((int(l), int(n)))


def spectral_matrix(m: int, n: int, sigma: np.ndarray, tag: int = 0) -> np.ndarray:
    """Dense m x n matrix with Haar singular vectors and the given singular
    values (len(sigma) <= min(m, n)), formed as (P * sigma) Q^T."""
    sigma = np.asarray(sigma, dtype=np.float64)
    P = haar(rng_for(W_FACTOR, 1, tag), m, sigma.size)
    Q = haar(rng_for(W_FACTOR, 2, tag), n, sigma.size)
    return np.ascontiguousarray((P * sigma) @ Q.T)

"""CPU oracle for low-precision rank compensation -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct FP64 implementation of what the GPU hot path
computes, written from the paper (El Mountasser & Jbilou, "Low-Precision Rank
Compensation for Matrices and Tensor Trains").  Only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it; it shares no
code with the GPU library and imports nothing from it.

The heavy loops live in ``lrc_oracle.c`` (plain C + OpenMP, no BLAS/LAPACK,
bitwise deterministic); this module strings them together in the paper's
order and notation.

Every function is pinned by a CPU test (``tests/test_oracle_*.py``) against
something other than itself: printed values of the paper's worked examples,
closed forms (Eckart-Young), library routines on special cases, brute force
on tiny inputs, and invariants.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# LRC_ORACLE_LIBRARY selects another build of the same C file (the sanitizer build)
_LIB_PATH = os.environ.get("LRC_ORACLE_LIBRARY") or os.path.join(_HERE, "liblrc_oracle.so")
_lib = None

PRECS = ("fp64", "fp32", "fp16")
BYTES = {"fp64": 8, "fp32": 4, "fp16": 2}   # b/8 for b bits per scalar (Sec. 4.2)

_dp = ctypes.POINTER(ctypes.c_double)
_i64p = ctypes.POINTER(ctypes.c_int64)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _build
        _build.build()
    lib = ctypes.CDLL(_LIB_PATH)
    i64, dbl, vp = ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
    lib.orc_round_f16.argtypes = [vp, vp, i64]
    lib.orc_round_f16.restype = i64
    lib.orc_round_f32.argtypes = [vp, vp, i64]
    lib.orc_round_f32.restype = i64
    lib.orc_f16_to_f64.argtypes = [vp, vp, i64]
    lib.orc_f16_to_f64.restype = None
    lib.orc_apply.argtypes = [vp, vp, vp, vp, vp, i64, i64, i64, i64]
    lib.orc_apply.restype = None
    lib.orc_lowrank_dense.argtypes = [vp, vp, vp, vp, i64, i64, i64]
    lib.orc_lowrank_dense.restype = None
    lib.orc_tt_chain.argtypes = [vp, vp, vp, ctypes.c_int, vp]
    lib.orc_tt_chain.restype = ctypes.c_int
    lib.orc_tt_entry.argtypes = [vp, vp, vp, ctypes.c_int, vp]
    lib.orc_tt_entry.restype = dbl
    lib.orc_sumsq.argtypes = [vp, i64]
    lib.orc_sumsq.restype = dbl
    lib.orc_sumsq_diff.argtypes = [vp, vp, i64]
    lib.orc_sumsq_diff.restype = dbl
    lib.orc_qr.argtypes = [vp, i64, i64, vp, vp]
    lib.orc_qr.restype = ctypes.c_int
    lib.orc_jacobi_svd.argtypes = [vp, i64, vp, vp, vp]
    lib.orc_jacobi_svd.restype = ctypes.c_int
    lib.orc_matmul.argtypes = [vp, vp, vp, i64, i64, i64]
    lib.orc_matmul.restype = None
    lib.orc_num_threads.argtypes = []
    lib.orc_num_threads.restype = ctypes.c_int
    lib.orc_set_num_threads.argtypes = [ctypes.c_int]
    lib.orc_set_num_threads.restype = None
    _lib = lib
    return lib


def _c(a: np.ndarray, dtype=np.float64) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=dtype)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops; results are independent of it."""
    _load().orc_set_num_threads(int(n))


# ---------------------------------------------------------------------------
# Rounding of stored values (Sec. 3.2; Remark after Thm 4.1; Sec. 4.3)
# ---------------------------------------------------------------------------

class OverflowInRounding(ArithmeticError):
    pass


def round_to(x: np.ndarray, prec: str, allow_overflow: bool = False) -> np.ndarray:
    """Round FP64 values to the storage format `prec` with a single
    round-to-nearest-even step (subnormals kept).  Returns an array of dtype
    float64 / float32 / float16 holding exactly the stored values."""
    lib = _load()
    x = _c(x)
    if prec == "fp64":
        return x.copy()
    if prec == "fp32":
        out = np.empty(x.shape, dtype=np.float32)
        ov = lib.orc_round_f32(_ptr(x), _ptr(out), x.size)
    elif prec == "fp16":
        bits = np.empty(x.shape, dtype=np.uint16)
        ov = lib.orc_round_f16(_ptr(x), _ptr(bits), x.size)
        out = bits.view(np.float16)
    else:
        raise ValueError(prec)
    if ov and not allow_overflow:
        raise OverflowInRounding(f"{ov} values overflow {prec}")
    return out


def widen(x: np.ndarray) -> np.ndarray:
    """Exact conversion of stored FP32/FP16 values to FP64."""
    lib = _load()
    if x.dtype == np.float16:
        bits = _c(x.view(np.uint16), np.uint16)
        out = np.empty(x.shape, dtype=np.float64)
        lib.orc_f16_to_f64(_ptr(bits), _ptr(out), x.size)
        return out
    return np.asarray(x, dtype=np.float64).copy()


def stored(x: np.ndarray, prec: str) -> np.ndarray:
    """The FP64 value of x after rounding to `prec` (round, then widen)."""
    return widen(round_to(x, prec))


# ---------------------------------------------------------------------------
# Matrix apply and dense reconstruction (Sec. 4.4 eq. gpu_matrix_apply)
# ---------------------------------------------------------------------------

def apply(U, s, V, X) -> np.ndarray:
    """Y = U diag(s) (V^T X) in FP64 with ascending sums (U m x k, V n x k,
    X n x b).  The paper writes the same product for a b x n batch as
    Y_p = [(X_p V) diag(s)] U^T; here X = X_p^T and Y = Y_p^T."""
    lib = _load()
    U, s, V, X = _c(U), _c(s), _c(V), _c(X)
    m, k = U.shape
    n, b = X.shape
    if V.shape != (n, k) or s.shape != (k,):
        raise ValueError("apply: shape mismatch")
    Y = np.empty((m, b))
    lib.orc_apply(_ptr(U), _ptr(s), _ptr(V), _ptr(X), _ptr(Y), m, n, k, b)
    return Y


def lowrank_dense(U, s, V) -> np.ndarray:
    """A_r = U diag(s) V^T in FP64 (Sec. 4, A_k = sum_j sigma_j u_j v_j^T)."""
    lib = _load()
    U, s, V = _c(U), _c(s), _c(V)
    m, k = U.shape
    n = V.shape[0]
    A = np.empty((m, n))
    lib.orc_lowrank_dense(_ptr(U), _ptr(s), _ptr(V), _ptr(A), m, n, k)
    return A


# ---------------------------------------------------------------------------
# Tensor-Train evaluation (Sec. 5.1; Sec. 7.5 eq. gpu_tt_reconstruction)
# ---------------------------------------------------------------------------

def tt_shape(cores):
    dims = [int(c.shape[1]) for c in cores]
    ranks = [int(cores[0].shape[0])] + [int(c.shape[2]) for c in cores]
    return dims, ranks


def _core_arrays(cores):
    cs = [_c(c) for c in cores]
    dims, ranks = tt_shape(cs)
    ptrs = (ctypes.c_void_p * len(cs))(*[c.ctypes.data for c in cs])
    return cs, dims, ranks, ptrs


def tt_full(cores) -> np.ndarray:
    """Dense FP64 tensor by the reshape chain B_l = Z_{l-1} K_l."""
    lib = _load()
    cs, dims, ranks, ptrs = _core_arrays(cores)
    if ranks[0] != 1 or ranks[-1] != 1:
        raise ValueError("boundary ranks must be 1")
    out = np.empty(int(np.prod(dims)))
    d = np.array(dims, dtype=np.int64)
    r = np.array(ranks, dtype=np.int64)
    rc = lib.orc_tt_chain(ptrs, _ptr(d), _ptr(r), len(cs), _ptr(out))
    if rc != 0:
        raise MemoryError("tt_full")
    return out.reshape(dims)


def tt_entry(cores, idx) -> float:
    """T(i_1..i_d) = G_1(i_1) G_2(i_2) ... G_d(i_d), one entry (0-based)."""
    lib = _load()
    cs, dims, ranks, ptrs = _core_arrays(cores)
    d = np.array(dims, dtype=np.int64)
    r = np.array(ranks, dtype=np.int64)
    ix = np.array(idx, dtype=np.int64)
    return float(lib.orc_tt_entry(ptrs, _ptr(d), _ptr(r), len(cs), _ptr(ix)))


def tt_storage_count(dims, ranks) -> int:
    """sum_l R_{l-1} n_l R_l (Sec. 5.1)."""
    return int(sum(int(ranks[l]) * int(dims[l]) * int(ranks[l + 1]) for l in range(len(dims))))


def tt_storage_bytes(dims, ranks, prec: str) -> int:
    return BYTES[prec] * tt_storage_count(dims, ranks)


def storage_bytes(m: int, n: int, k: int, prec: str) -> int:
    """Stored bytes of a rank-k SVD representation: (b/8) k (m+n+1) (Sec. 4.2)."""
    return BYTES[prec] * int(k) * (int(m) + int(n) + 1)


# ---------------------------------------------------------------------------
# Norms
# ---------------------------------------------------------------------------

def fro(a) -> float:
    a = _c(a)
    return math.sqrt(_load().orc_sumsq(_ptr(a), a.size))


def fro_diff(a, b) -> float:
    a, b = _c(a), _c(b)
    if a.size != b.size:
        raise ValueError("fro_diff: size mismatch")
    return math.sqrt(_load().orc_sumsq_diff(_ptr(a), _ptr(b), a.size))


def tail_norms(sigma) -> np.ndarray:
    """E[k] = (sum_{j>k} sigma_j^2)^{1/2} for k = 0..p (Sec. 4, Eckart-Young),
    all from one reverse cumulative FP64 sum, so E is non-increasing."""
    s = np.asarray(sigma, dtype=np.float64)
    p = len(s)
    E = np.zeros(p + 1)
    acc = 0.0
    for j in range(p - 1, -1, -1):
        acc += float(s[j]) * float(s[j])
        E[j] = math.sqrt(acc)
    return E


# ---------------------------------------------------------------------------
# Offline factorizations: Householder QR, one-sided Jacobi SVD, TT-SVD
# ---------------------------------------------------------------------------

def matmul(A, B) -> np.ndarray:
    lib = _load()
    A, B = _c(A), _c(B)
    m, p = A.shape
    p2, n = B.shape
    if p != p2:
        raise ValueError("matmul shape")
    C = np.empty((m, n))
    lib.orc_matmul(_ptr(A), _ptr(B), _ptr(C), m, p, n)
    return C


def qr(A):
    """Thin Householder QR, A = Q R with diag(R) >= 0 (m >= n)."""
    lib = _load()
    A = _c(A)
    m, n = A.shape
    Q = np.empty((m, n))
    R = np.empty((n, n))
    if lib.orc_qr(_ptr(A), m, n, _ptr(Q), _ptr(R)) != 0:
        raise ValueError("qr: need m >= n")
    return Q, R


def svd(A):
    """Thin SVD A = U diag(S) Vt by QR preconditioning and one-sided Jacobi
    on the triangular factor; S non-increasing; the largest-magnitude entry
    of every column of U is positive."""
    lib = _load()
    A = _c(A)
    m, n = A.shape
    if m < n:
        U2, S, Vt2 = svd(A.T)
        U, Vt = Vt2.T.copy(), U2.T.copy()
    else:
        Q, R = qr(A)
        Ur = np.empty((n, n))
        S = np.empty(n)
        Vr = np.empty((n, n))
        if lib.orc_jacobi_svd(_ptr(R), n, _ptr(Ur), _ptr(S), _ptr(Vr)) < 0:
            raise ArithmeticError("Jacobi SVD did not converge")
        U = matmul(Q, Ur)
        Vt = Vr.T.copy()
    # sign convention on the final U
    for j in range(U.shape[1]):
        col = U[:, j]
        i = int(np.argmax(np.abs(col)))
        if col[i] < 0:
            U[:, j] = -col
            Vt[j, :] = -Vt[j, :]
    return U, S, Vt


def tt_svd(T: np.ndarray, ranks=None, eps=None, svd_memo=None):
    """TT-SVD (Oseledets 2011, as used in Sec. 5.1): sequential truncated
    SVDs of the unfoldings.  Either fixed nominal ranks (each capped by the
    valid unfolding dimension, min(R_nom, r_{l-1} n_l, prod_{i>l} n_i), as in
    Sec. 7.4) or a relative tolerance eps with per-step threshold
    eps ||T||_F / sqrt(d-1).  Returns FP64 cores r_{l-1} x n_l x r_l.

    svd_memo: optional dict shared by several runs on the same tensor.  The
    unfolding of step l depends only on the ranks kept before it, so its SVD
    is stored under that rank prefix and reused (the first unfolding's SVD is
    the same for every rank choice); the cores are bit for bit those of a run
    without the memo."""
    dims = [int(x) for x in T.shape]
    d = len(dims)
    if (ranks is None) == (eps is None):
        raise ValueError("give exactly one of ranks / eps")
    if ranks is not None:
        ranks = [int(r) for r in (ranks if np.ndim(ranks) else [ranks] * (d - 1))]
        if len(ranks) != d - 1:
            raise ValueError("need d-1 ranks")
    delta = None
    if eps is not None:
        delta = float(eps) * fro(T) / math.sqrt(d - 1)
    C = _c(T).reshape(dims[0], -1)
    r_prev = 1
    cores = []
    kept = ()
    for l in range(d - 1):
        C = C.reshape(r_prev * dims[l], -1)
        if svd_memo is not None and kept in svd_memo:
            U, S, Vt = svd_memo[kept]
        else:
            U, S, Vt = svd(C)
            if svd_memo is not None:
                svd_memo[kept] = (U, S, Vt)
        cap = min(C.shape)
        if ranks is not None:
            r = min(ranks[l], cap)
        else:
            tails = tail_norms(S)
            r = cap
            for cand in range(1, cap + 1):
                if tails[cand] <= delta:
                    r = cand
                    break
        cores.append(np.ascontiguousarray(U[:, :r].reshape(r_prev, dims[l], r)))
        C = S[:r, None] * Vt[:r, :]
        r_prev = r
        kept = kept + (r,)
    cores.append(np.ascontiguousarray(C.reshape(r_prev, dims[-1], 1)))
    return cores


def left_orthogonalize(cores):
    """Left-orthogonal gauge (Sec. 6.1; Algorithm alg:tt_compensation step 3):
    for l = 1..d-1, QR of the left unfolding (r_{l-1} n_l) x r_l with
    diag(R) >= 0, keep Q as core l and absorb R into core l+1."""
    cs = [np.array(c, dtype=np.float64) for c in cores]
    d = len(cs)
    for l in range(d - 1):
        r0, n, r1 = cs[l].shape
        M = cs[l].reshape(r0 * n, r1)
        if r0 * n < r1:
            raise ValueError("left_orthogonalize: rank exceeds the unfolding dimension")
        Q, R = qr(M)
        cs[l] = np.ascontiguousarray(Q.reshape(r0, n, r1))
        nxt = cs[l + 1]
        cs[l + 1] = np.ascontiguousarray(matmul(R, nxt.reshape(r1, -1)).reshape(nxt.shape))
    return cs


def round_cores(cores, prec: str):
    """Stored cores: each entry rounded individually (Algorithm step 4)."""
    return [round_to(c, prec) for c in cores]


# ---------------------------------------------------------------------------
# Certificates (Thm thm:matrix_rank_compensation; Thm thm:tt_conditional;
# Algorithm alg:tt_compensation; outcome vocabulary of Sec. 4.1)
# ---------------------------------------------------------------------------

def _outcome(certified: bool, mem_win: bool) -> int:
    """Algorithm alg:tt_compensation: 2 = certified non-increase and memory
    win, 1 = certified accuracy non-increase only, 0 = fall back to FP64."""
    if certified and mem_win:
        return 2
    if certified:
        return 1
    return 0


def matrix_certificate(sigma, U, s, V, k: int, prec: str, A=None):
    """Matrix rank compensation, k -> k+1 (Thm thm:matrix_rank_compensation).

    sigma: all singular values of A (non-increasing); U (m x (k+1)),
    s (k+1), V (n x (k+1)): the FP64 rank-(k+1) factors.  A_hat is formed by
    rounding U, s and V individually to `prec` and contracting in FP64
    (Remark after the theorem).  E_k and E_{k+1} come from the spectrum
    (Eckart-Young); eta = ||A_{k+1} - A_hat||_F; the verdict is the direct
    form E_{k+1} + eta <= E_k, an exact FP64 comparison."""
    U, s, V = _c(U), _c(s), _c(V)
    m, r = U.shape
    n = V.shape[0]
    if r != k + 1:
        raise ValueError("factors must have rank k+1")
    E = tail_norms(sigma)
    Ek, Ek1 = float(E[k]), float(E[k + 1])
    norm_ref = float(E[0])
    Uh, sh, Vh = stored(U, prec), stored(s, prec), stored(V, prec)
    A_aug = lowrank_dense(U, s, V)
    A_hat = lowrank_dense(Uh, sh, Vh)
    eta = fro_diff(A_aug, A_hat)
    err_new = fro_diff(A, A_hat) if A is not None else float("nan")
    del A_aug, A_hat
    gain = float(sigma[k]) ** 2
    certified = (Ek1 + eta) <= Ek
    bytes_base = storage_bytes(m, n, k, "fp64")
    bytes_aug = storage_bytes(m, n, k + 1, prec)
    mem_win = bytes_aug < bytes_base
    acc_nonincrease = (err_new <= Ek) if A is not None else False
    acc_win = (err_new < Ek) if A is not None else False
    return dict(E_base=Ek, E_aug=Ek1, eta=eta, err_new=err_new, gain=gain,
                margin=Ek - Ek1 - eta, norm_ref=norm_ref,
                bytes_base=bytes_base, bytes_aug=bytes_aug,
                certified=bool(certified), acc_nonincrease=bool(acc_nonincrease),
                acc_win=bool(acc_win), mem_win=bool(mem_win),
                practical_win=bool(acc_win and mem_win),
                outcome=_outcome(certified, mem_win))


def tt_certificate(T, base_cores, aug_cores, prec: str):
    """Conditional TT rank compensation (Thm thm:tt_conditional) for given
    FP64 base cores (rank R) and FP64 augmented cores (rank R+, already in
    the left-orthogonal gauge), Algorithm alg:tt_compensation steps 4-9:
    round the augmented cores, measure E_R, E_{R+}, S_TT, eta_TT by FP64
    reconstruction, then decide."""
    dims = list(T.shape)
    _, rb = tt_shape(base_cores)
    _, ra = tt_shape(aug_cores)
    aug_h = [widen(c) for c in round_cores(aug_cores, prec)]
    T_R = tt_full(base_cores)
    T_Rp = tt_full(aug_cores)
    T_h = tt_full(aug_h)
    E_R = fro_diff(T, T_R)
    E_Rp = fro_diff(T, T_Rp)
    eta = fro_diff(T_Rp, T_h)
    err_new = fro_diff(T, T_h)
    norm_ref = fro(T)
    bytes_base = tt_storage_bytes(dims, rb, "fp64")
    bytes_aug = tt_storage_bytes(dims, ra, prec)
    certified = (E_Rp + eta) <= E_R
    mem_win = bytes_aug < bytes_base
    return dict(E_base=E_R, E_aug=E_Rp, eta=eta, err_new=err_new,
                gain=E_R * E_R - E_Rp * E_Rp, margin=E_R - E_Rp - eta,
                norm_ref=norm_ref, bytes_base=bytes_base, bytes_aug=bytes_aug,
                certified=bool(certified), acc_nonincrease=bool(err_new <= E_R),
                acc_win=bool(err_new < E_R), mem_win=bool(mem_win),
                practical_win=bool(err_new < E_R and mem_win),
                outcome=_outcome(certified, mem_win),
                ranks_base=rb, ranks_aug=ra)


def tt_compensation(T, R=None, R_plus=None, prec: str = "fp16", eps=None, delta=None):
    """Algorithm alg:tt_compensation end to end.  Base ranks come from
    nominal ranks R (capped) or from a TT-SVD tolerance eps; the augmented
    run is a separate TT-SVD at R_plus (or at the base ranks + delta), then
    left-orthogonalized, rounded and certified."""
    base = tt_svd(T, ranks=R) if eps is None else tt_svd(T, eps=eps)
    _, rb = tt_shape(base)
    if R_plus is None:
        R_plus = [r + int(delta) for r in rb[1:-1]]
    aug = left_orthogonalize(tt_svd(T, ranks=R_plus))
    res = tt_certificate(T, base, aug, prec)
    res["base_cores"], res["aug_cores"] = base, aug
    return res


# ---------------------------------------------------------------------------
# Fixed-memory comparison (Sec. sec:hyperspectral_application): quality
# measures of a reconstruction and the memory-matched FP64 rank.
# ---------------------------------------------------------------------------

def band_range(xb) -> float:
    """L_b of one reference band: max - min, or max(max|X_b|, 1) for a
    constant band."""
    lo, hi = float(np.min(xb)), float(np.max(xb))
    if hi > lo:
        return hi - lo
    return max(max(abs(lo), abs(hi)), 1.0)


def band_quality(X, Xh) -> dict:
    """Quality of Xh against the reference X, both FP64 with the spectral
    bands along the last axis and the pixels along the others:
      rel_err  ||X - Xh||_F / ||X||_F
      psnr     mean over bands of 20 log10(L_b / sqrt(MSE_b))
      ssim     mean over bands of the SSIM variant evaluated once per whole
               band with population means, variances and covariance,
               C1 = (0.01 L_b)^2, C2 = (0.03 L_b)^2
      sam      mean over pixels with ||x|| ||xh|| > 0 of the angle between
               the reference and reconstructed spectra (radians)."""
    X = np.asarray(X, dtype=np.float64)
    Xh = np.asarray(Xh, dtype=np.float64)
    B = X.shape[-1]
    Xm = X.reshape(-1, B)
    Ym = Xh.reshape(-1, B)
    psnr, ssim = [], []
    for b in range(B):
        x, y = Xm[:, b], Ym[:, b]
        L = band_range(x)
        mse = float(np.mean((x - y) ** 2))
        with np.errstate(divide="ignore"):
            psnr.append(20.0 * math.log10(L / math.sqrt(mse)) if mse > 0 else math.inf)
        mx, my = float(np.mean(x)), float(np.mean(y))
        vx, vy = float(np.mean((x - mx) ** 2)), float(np.mean((y - my) ** 2))
        cxy = float(np.mean((x - mx) * (y - my)))
        c1, c2 = (0.01 * L) ** 2, (0.03 * L) ** 2
        ssim.append((2 * mx * my + c1) * (2 * cxy + c2) / ((mx * mx + my * my + c1) * (vx + vy + c2)))
    nx = np.sqrt(np.sum(Xm * Xm, axis=1))
    ny = np.sqrt(np.sum(Ym * Ym, axis=1))
    keep = nx * ny > 0
    cos = np.sum(Xm * Ym, axis=1)[keep] / (nx[keep] * ny[keep])
    angles = np.arccos(np.clip(cos, -1.0, 1.0))
    return dict(rel_err=fro_diff(X, Xh) / fro(X), psnr=float(np.mean(psnr)), ssim=float(np.mean(ssim)),
                sam=float(np.mean(angles)) if angles.size else math.nan, sam_pixels=int(np.count_nonzero(keep)))


def capped_ranks(dims, nominal):
    """Uniform nominal TT ranks capped by the unfolding dimensions,
    r_l <= min(R, r_{l-1} n_l, prod_{i>l} n_i) (Sec. 7.4)."""
    ranks = [1]
    for l in range(len(dims) - 1):
        ranks.append(int(min(int(nominal), ranks[-1] * int(dims[l]), int(np.prod([int(n) for n in dims[l + 1:]])))))
    return ranks + [1]


def memory_matched_rank(dims, budget_bytes: int):
    """The largest uniform FP64 TT rank (capped as above) whose exact TT
    storage does not exceed budget_bytes, with its rank vector; (0, None)
    if even rank 1 does not fit (Sec. sec:hyperspectral_application)."""
    best = (0, None)
    R = 1
    while True:
        ranks = capped_ranks(dims, R)
        if tt_storage_bytes(dims, ranks, "fp64") > budget_bytes:
            return best
        best = (R, ranks)
        if ranks == capped_ranks(dims, R + 1):   # every rank capped: storage stops growing
            return best
        R += 1


# ---------------------------------------------------------------------------
# Randomized factorizations (the end-to-end decomposition that Sec.
# sec:conclusion leaves to future work).  The paper fixes no GPU method for
# it; these follow the randomized range finder of Halko, Martinsson and Tropp
# (SIAM Review 2011: Gaussian sketch, optional subspace iterations with
# re-orthonormalization, then the exact SVD of the small projected matrix),
# and TT-SVD (Sec. 5.1) with every truncated SVD replaced by that.  The
# Gaussian test vectors are inputs: the caller draws them.
# ---------------------------------------------------------------------------

def randomized_svd(A, Omega, k: int, power_iters: int = 0):
    """Rank-k randomized SVD of A (m x n) with the l test vectors given as
    the rows of Omega (l x n), k <= l <= min(m, n):
      Y = A Omega^T, Q = orth(Y);  q times: Q = orth(A orth(A^T Q));
      B = Q^T A = Ub S Vt (exact SVD);  U = Q Ub[:, :k].
    Returns U (m x k), S (k), Vt (k x n).  U diag(S) Vt = Q_k Q_k^T A with
    Q_k = U: an orthogonal projection of A's columns."""
    A = _c(A)
    Om = _c(Omega)
    m, n = A.shape
    l = Om.shape[0]
    if Om.shape[1] != n or not (1 <= k <= l <= min(m, n)):
        raise ValueError("randomized_svd: need Omega l x n with k <= l <= min(m, n)")
    Q, _ = qr(matmul(A, Om.T))
    for _ in range(int(power_iters)):
        Z, _ = qr(matmul(A.T, Q))
        Q, _ = qr(matmul(A, Z))
    B = matmul(Q.T, A)
    Ub, S, Vt = svd(B)
    return matmul(Q, Ub[:, :k]), S[:k].copy(), np.ascontiguousarray(Vt[:k])


def tt_svd_randomized(T: np.ndarray, ranks, omegas, power_iters: int = 0):
    """TT-SVD (Sec. 5.1) with the truncated SVD of unfolding l replaced by
    randomized_svd(C_l, omegas[l], ranks[l]); C_l is (r_{l-1} n_l) x
    prod_{i>l} n_i and omegas[l] holds l_l test vectors of that length as
    rows.  Ranks are used as given (r_l <= l_l <= both unfolding sizes).
    Returns the FP64 cores and, per step, the r_l singular values kept and
    the step's truncation error eps_l = ||C_l - U S Vt||_F (the terms of
    eq. tt_svd_error)."""
    dims = [int(x) for x in T.shape]
    d = len(dims)
    ranks = [int(r) for r in ranks]
    if len(ranks) != d - 1 or len(omegas) != d - 1:
        raise ValueError("need d-1 ranks and test matrices")
    C = _c(T).reshape(dims[0], -1)
    r_prev = 1
    cores, sigma, step_err = [], [], []
    for l in range(d - 1):
        C = C.reshape(r_prev * dims[l], -1)
        U, S, Vt = randomized_svd(C, omegas[l], ranks[l], power_iters)
        r = ranks[l]
        nxt = S[:, None] * Vt
        step_err.append(fro_diff(C, matmul(U, nxt)))
        sigma.append(S)
        cores.append(np.ascontiguousarray(U.reshape(r_prev, dims[l], r)))
        C = nxt
        r_prev = r
    cores.append(np.ascontiguousarray(C.reshape(r_prev, dims[-1], 1)))
    return cores, {"sigma": sigma, "step_err": step_err}

"""Python binding of the rank-compensation hot path (liblrc.so, gfx950).

Argument marshalling only: torch tensors are checked for device, dtype and
layout, their data pointers and torch's current stream are passed to the C
ABI declared in include/lrc.h, and every computation runs in the library's
HIP kernels.  There is no CPU fallback: if the library is missing this
module raises on first use.

Precision follows the tensors' dtype: float64 -> FP64, float32 -> FP32,
float16 -> FP16 (FP32 accumulation).
"""
from __future__ import annotations

import ctypes
import math
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
# LRC_LIBRARY selects another build of the same sources (the host-sanitized build)
LIB_PATH = os.environ.get("LRC_LIBRARY") or os.path.join(HERE, "liblrc.so")
HEADER = os.path.join(os.path.dirname(HERE), "include", "lrc.h")

FP64, FP32, FP16 = 0, 1, 2
PATH_AUTO, PATH_STREAM, PATH_MFMA = 0, 1, 2
CERT_MATRIX, CERT_TT = 0, 1
ERRORS = {-1: "EINVAL", -2: "EOVERFLOW", -3: "EHIP", -4: "ENOMEM", -5: "ENODEV", -6: "ENUMERIC"}
PREC_NAMES = {"fp64": FP64, "fp32": FP32, "fp16": FP16}


class LrcError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{ERRORS.get(code, code)}: {msg}")
        self.code = code


_i64 = ctypes.c_int64
_vp = ctypes.c_void_p


class CertArgs(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int), ("prec", ctypes.c_int),
        ("m", _i64), ("n", _i64), ("k", _i64),
        ("sigma", ctypes.POINTER(ctypes.c_double)), ("n_sigma", _i64),
        ("U", _vp), ("s", _vp), ("V", _vp),
        ("Uh", _vp), ("sh", _vp), ("Vh", _vp),
        ("A", _vp),
        ("d", ctypes.c_int),
        ("dims", ctypes.POINTER(_i64)),
        ("T", _vp),
        ("ranks_base", ctypes.POINTER(_i64)), ("cores_base", ctypes.POINTER(_vp)),
        ("ranks_aug", ctypes.POINTER(_i64)), ("cores_aug", ctypes.POINTER(_vp)),
        ("cores_aug_h", ctypes.POINTER(_vp)),
    ]


class CertResult(ctypes.Structure):
    _fields_ = [
        ("E_base", ctypes.c_double), ("E_aug", ctypes.c_double), ("eta", ctypes.c_double),
        ("err_new", ctypes.c_double), ("gain", ctypes.c_double), ("margin", ctypes.c_double),
        ("norm_ref", ctypes.c_double),
        ("bytes_base", _i64), ("bytes_aug", _i64),
        ("certified", ctypes.c_int), ("acc_nonincrease", ctypes.c_int), ("acc_win", ctypes.c_int),
        ("mem_win", ctypes.c_int), ("practical_win", ctypes.c_int), ("outcome", ctypes.c_int),
    ]


class Quality(ctypes.Structure):
    _fields_ = [("rel_err", ctypes.c_double), ("psnr", ctypes.c_double), ("ssim", ctypes.c_double),
                ("sam", ctypes.c_double), ("sam_pixels", _i64), ("pixels", _i64), ("bands", _i64)]


_lib = None


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_12969_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    L.lrc_matrix_apply.argtypes = [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, ctypes.c_int]
    L.lrc_matrix_apply.restype = ctypes.c_int
    L.lrc_matrix_apply_noalloc.argtypes = [_vp, _vp, _vp, _vp, _vp, _i64, _i64, _i64, _i64, ctypes.c_int]
    L.lrc_matrix_apply_noalloc.restype = ctypes.c_int
    L.lrc_mfma_ceiling.argtypes = [ctypes.c_int, ctypes.POINTER(ctypes.c_double)]
    L.lrc_mfma_ceiling.restype = ctypes.c_int
    L.lrc_matrix_apply_path.argtypes = [_i64, _i64, _i64, _i64, ctypes.c_int]
    L.lrc_matrix_apply_path.restype = ctypes.c_int
    L.lrc_set_apply_path.argtypes = [ctypes.c_int]
    L.lrc_set_apply_path.restype = ctypes.c_int
    L.lrc_tt_reconstruct.argtypes = [ctypes.POINTER(_vp), ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                                     ctypes.c_int, _vp, ctypes.c_int]
    L.lrc_tt_reconstruct.restype = ctypes.c_int
    L.lrc_certify.argtypes = [ctypes.POINTER(CertArgs), ctypes.POINTER(CertResult)]
    L.lrc_certify.restype = ctypes.c_int
    L.lrc_round.argtypes = [_vp, _vp, _i64, ctypes.c_int, ctypes.POINTER(_i64)]
    L.lrc_round.restype = ctypes.c_int
    L.lrc_tt_left_orthogonalize.argtypes = [ctypes.POINTER(_vp), ctypes.POINTER(_i64), ctypes.POINTER(_i64),
                                            ctypes.c_int]
    L.lrc_tt_left_orthogonalize.restype = ctypes.c_int
    L.lrc_band_quality.argtypes = [_vp, _vp, _i64, _i64, ctypes.c_int, ctypes.c_double, ctypes.POINTER(Quality)]
    L.lrc_band_quality.restype = ctypes.c_int
    L.lrc_tt_quality.argtypes = [ctypes.POINTER(_vp), ctypes.POINTER(_i64), ctypes.POINTER(_i64), ctypes.c_int,
                                 ctypes.c_int, _vp, ctypes.c_double, ctypes.POINTER(Quality)]
    L.lrc_tt_quality.restype = ctypes.c_int
    L.lrc_tt_memory_matched_rank.argtypes = [ctypes.POINTER(_i64), ctypes.c_int, _i64, ctypes.POINTER(_i64)]
    L.lrc_tt_memory_matched_rank.restype = _i64
    L.lrc_rsvd.argtypes = [_vp, _i64, _i64, _vp, _i64, ctypes.c_int, _i64, _vp, _vp, _vp]
    L.lrc_rsvd.restype = ctypes.c_int
    L.lrc_tt_rsvd.argtypes = [_vp, ctypes.POINTER(_i64), ctypes.POINTER(_i64), ctypes.c_int, ctypes.POINTER(_vp),
                              ctypes.POINTER(_i64), ctypes.c_int, ctypes.POINTER(_vp), _vp]
    L.lrc_tt_rsvd.restype = ctypes.c_int
    L.lrc_storage_bytes.argtypes = [_i64, _i64, _i64, ctypes.c_int]
    L.lrc_storage_bytes.restype = _i64
    L.lrc_tt_storage_bytes.argtypes = [ctypes.POINTER(_i64), ctypes.POINTER(_i64), ctypes.c_int, ctypes.c_int]
    L.lrc_tt_storage_bytes.restype = _i64
    L.lrc_set_stream.argtypes = [_vp]
    L.lrc_set_stream.restype = ctypes.c_int
    L.lrc_last_error.argtypes = []
    L.lrc_last_error.restype = ctypes.c_char_p
    L.lrc_shutdown.argtypes = []
    L.lrc_shutdown.restype = None
    L.lrc_version.argtypes = []
    L.lrc_version.restype = ctypes.c_int
    L.lrc_profile_enable.argtypes = [ctypes.c_int]
    L.lrc_profile_enable.restype = ctypes.c_int
    L.lrc_profile_filter.argtypes = [ctypes.c_char_p]
    L.lrc_profile_filter.restype = ctypes.c_int
    L.lrc_profile_reset.argtypes = []
    L.lrc_profile_reset.restype = None
    L.lrc_profile_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(_i64), ctypes.POINTER(ctypes.c_double)]
    L.lrc_profile_read.restype = ctypes.c_int
    L.lrc_profile_labels.argtypes = [ctypes.c_char_p, _i64]
    L.lrc_profile_labels.restype = _i64
    _lib = L
    return L


def header_symbols():
    """Function names declared in include/lrc.h."""
    with open(HEADER) as fh:
        text = fh.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]*?\b(lrc_\w+)\s*\(", text, flags=re.M)))


def _check(rc: int):
    if rc < 0:
        raise LrcError(rc, lib().lrc_last_error().decode())
    return rc


def _prec_of(t) -> int:
    import torch
    m = {torch.float64: FP64, torch.float32: FP32, torch.float16: FP16}
    if t.dtype not in m:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return m[t.dtype]


def _dev(*ts):
    for t in ts:
        if not t.is_cuda:
            raise ValueError("tensors must be on the GPU")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous (row-major)")


def _bind_stream(device=None):
    import torch
    st = torch.cuda.current_stream(device)
    lib().lrc_set_stream(_vp(st.cuda_stream))


# ------------------------------------------------------------------ API ---

def storage_bytes(m: int, n: int, k: int, prec) -> int:
    p = PREC_NAMES.get(prec, prec)
    return _check(lib().lrc_storage_bytes(m, n, k, p))


def tt_storage_bytes(dims, ranks, prec) -> int:
    p = PREC_NAMES.get(prec, prec)
    d = len(dims)
    D = (_i64 * d)(*dims)
    R = (_i64 * (d + 1))(*ranks)
    return _check(lib().lrc_tt_storage_bytes(D, R, d, p))


def apply_path(m: int, n: int, k: int, batch: int, prec) -> int:
    p = PREC_NAMES.get(prec, prec)
    return _check(lib().lrc_matrix_apply_path(m, n, k, batch, p))


def set_apply_path(path: int):
    _check(lib().lrc_set_apply_path(path))


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def matrix_apply(U, s, V, X, Y=None):
    """Y = U diag(s) (V^T X): U (m x k), s (k), V (n x k), X (n x batch).
    A caller-supplied Y must be (m, batch), of U's dtype and on U's device."""
    import torch
    prec = _prec_of(U)
    for t in (s, V, X):
        if t.dtype != U.dtype:
            raise TypeError("all factors and the batch must share one dtype")
    _need(U.dim() == 2 and X.dim() == 2, "U and X must be matrices")
    m, k = U.shape
    n, b = X.shape
    _need(tuple(V.shape) == (n, k) and tuple(s.shape) == (k,),
          f"shape mismatch: V {tuple(V.shape)} (want {(n, k)}), s {tuple(s.shape)} (want {(k,)})")
    if Y is not None:
        _need(tuple(Y.shape) == (m, b), f"Y has shape {tuple(Y.shape)}, want {(m, b)}")
        _need(Y.dtype == U.dtype, f"Y has dtype {Y.dtype}, want {U.dtype}")
    _dev(U, s, V, X)
    if Y is None:
        Y = torch.empty((m, b), dtype=U.dtype, device=U.device)
    _dev(Y)
    _need(all(t.device == U.device for t in (s, V, X, Y)), "all tensors must be on one device")
    _bind_stream(U.device)
    _check(lib().lrc_matrix_apply(U.data_ptr(), s.data_ptr(), V.data_ptr(), X.data_ptr(), Y.data_ptr(),
                                  m, n, k, b, prec))
    return Y


def tt_shape(cores):
    dims = [int(c.shape[1]) for c in cores]
    ranks = [int(cores[0].shape[0])] + [int(c.shape[2]) for c in cores]
    return dims, ranks


def matrix_apply_noalloc(U, s, V, X, Y):
    """matrix_apply through the allocation-free entry point: Y (m x batch)
    must be supplied; the library's per-device scratch array holds the
    intermediate sums (calls overlapping on one device race on it)."""
    prec = _prec_of(U)
    for t in (s, V, X, Y):
        if t.dtype != U.dtype:
            raise TypeError("all factors, the batch and Y must share one dtype")
    _need(U.dim() == 2 and X.dim() == 2, "U and X must be matrices")
    m, k = U.shape
    n, b = X.shape
    _need(tuple(V.shape) == (n, k) and tuple(s.shape) == (k,), "shape mismatch")
    _need(tuple(Y.shape) == (m, b), f"Y has shape {tuple(Y.shape)}, want {(m, b)}")
    _dev(U, s, V, X, Y)
    _bind_stream(U.device)
    _check(lib().lrc_matrix_apply_noalloc(U.data_ptr(), s.data_ptr(), V.data_ptr(), X.data_ptr(), Y.data_ptr(),
                                          m, n, k, b, prec))
    return Y


def _check_train(cores):
    """Consistent TT cores: 3-D (r_{l-1}, n_l, r_l), adjacent ranks equal,
    boundary ranks 1, one dtype."""
    _need(len(cores) >= 1, "need at least one core")
    for l, c in enumerate(cores):
        _need(c.dim() == 3, f"core {l} must be 3-D (r_prev, n, r_next)")
        if c.dtype != cores[0].dtype:
            raise TypeError("all cores must share one dtype")
        if l > 0:
            _need(int(c.shape[0]) == int(cores[l - 1].shape[2]),
                  f"core {l} starts with rank {int(c.shape[0])}, core {l - 1} ends with {int(cores[l - 1].shape[2])}")
    _need(int(cores[0].shape[0]) == 1 and int(cores[-1].shape[2]) == 1, "boundary ranks must be 1")


def tt_reconstruct(cores, out=None):
    """Dense tensor (C order) from TT cores G_l of shape (r_{l-1}, n_l, r_l).
    A caller-supplied `out` must hold prod(dims) entries of the cores'
    dtype on their device."""
    import torch
    prec = _prec_of(cores[0])
    _check_train(cores)
    dims, ranks = tt_shape(cores)
    d = len(cores)
    if out is not None:
        _need(out.numel() == math.prod(dims), f"out has {out.numel()} entries, want {math.prod(dims)}")
        _need(out.dtype == cores[0].dtype, f"out has dtype {out.dtype}, want {cores[0].dtype}")
    _dev(*cores)
    if out is None:
        out = torch.empty(dims, dtype=cores[0].dtype, device=cores[0].device)
    _dev(out)
    _need(all(c.device == out.device for c in cores), "cores and out must be on one device")
    ptrs = (_vp * d)(*[c.data_ptr() for c in cores])
    D = (_i64 * d)(*dims)
    R = (_i64 * (d + 1))(*ranks)
    _bind_stream(cores[0].device)
    _check(lib().lrc_tt_reconstruct(ptrs, D, R, d, out.data_ptr(), prec))
    return out


def round_to(x, prec, out=None, count_overflow: bool = False):
    """Stored values of a float64 tensor: one round-to-nearest-even step to
    `prec` ("fp32" / "fp16", or a torch dtype).  Returns the rounded tensor,
    and with count_overflow=True also the number of finite values that
    became infinite (this waits for the result)."""
    import torch
    _dev(x)
    if x.dtype != torch.float64:
        raise TypeError("x must be float64")
    dt = {"fp64": torch.float64, "fp32": torch.float32, "fp16": torch.float16}.get(prec, prec)
    p = {torch.float64: FP64, torch.float32: FP32, torch.float16: FP16}[dt]
    if out is None:
        out = torch.empty(x.shape, dtype=dt, device=x.device)
    _dev(out)
    if out.dtype != dt or out.numel() != x.numel():
        raise ValueError("out must have the target dtype and x's size")
    _bind_stream(x.device)
    n = _i64(0)
    _check(lib().lrc_round(x.data_ptr(), out.data_ptr(), x.numel(), p, ctypes.byref(n) if count_overflow else None))
    return (out, int(n.value)) if count_overflow else out


def tt_left_orthogonalize(cores):
    """Left-orthogonal gauge of float64 TT cores (r_{l-1}, n_l, r_l), in
    place; returns the same list."""
    import torch
    _dev(*cores)
    for c in cores:
        if c.dtype != torch.float64:
            raise TypeError("the gauge takes float64 cores")
    dims, ranks = tt_shape(cores)
    d = len(cores)
    ptrs = (_vp * d)(*[c.data_ptr() for c in cores])
    D = (_i64 * d)(*dims)
    R = (_i64 * (d + 1))(*ranks)
    _bind_stream(cores[0].device)
    _check(lib().lrc_tt_left_orthogonalize(ptrs, D, R, d))
    return cores


def _quality(q: Quality) -> dict:
    return {f: getattr(q, f) for f, _ in Quality._fields_}


def band_quality(X, Xh, scale: float = 1.0) -> dict:
    """Quality of Xh (any storage dtype) against the float64 reference X,
    bands along the last axis (relative error, mean band PSNR, mean band
    SSIM variant, mean spectral angle)."""
    import torch
    _dev(X, Xh)
    if X.dtype != torch.float64 or X.shape != Xh.shape or X.dim() < 2:
        raise ValueError("X must be float64 with at least two axes, Xh of the same shape")
    B = int(X.shape[-1])
    _bind_stream(X.device)
    q = Quality()
    _check(lib().lrc_band_quality(X.data_ptr(), Xh.data_ptr(), X.numel() // B, B, _prec_of(Xh), float(scale),
                                  ctypes.byref(q)))
    return _quality(q)


def tt_quality(cores, X, scale: float = 1.0) -> dict:
    """Quality of the FP64 contraction of the stored cores (times scale)
    against the float64 reference X of the full tensor shape."""
    import torch
    _dev(*cores, X)
    if X.dtype != torch.float64:
        raise TypeError("X must be float64")
    dims, ranks = tt_shape(cores)
    if list(X.shape) != dims:
        raise ValueError("X must have the tensor's shape")
    d = len(cores)
    ptrs = (_vp * d)(*[c.data_ptr() for c in cores])
    D = (_i64 * d)(*dims)
    R = (_i64 * (d + 1))(*ranks)
    _bind_stream(X.device)
    q = Quality()
    _check(lib().lrc_tt_quality(ptrs, D, R, d, _prec_of(cores[0]), X.data_ptr(), float(scale), ctypes.byref(q)))
    return _quality(q)


def memory_matched_rank(dims, budget_bytes: int):
    """(R, capped rank vector) of the largest uniform FP64 TT rank within
    budget_bytes; (0, None) if rank 1 does not fit."""
    d = len(dims)
    D = (_i64 * d)(*dims)
    out = (_i64 * (d + 1))()
    R = _check(lib().lrc_tt_memory_matched_rank(D, d, int(budget_bytes), out))
    return (int(R), [int(v) for v in out]) if R > 0 else (0, None)


def rsvd(A, omega, k: int, power_iters: int = 0):
    """Rank-k randomized SVD of the float64 device matrix A (m x n) with the
    test vectors as the rows of omega (l x n): returns U (m x k), s (k),
    V (n x k), float64 on A's device, with U diag(s) V^T = U U^T A."""
    import torch
    _dev(A, omega)
    if A.dtype != torch.float64 or omega.dtype != torch.float64 or A.dim() != 2 or omega.dim() != 2:
        raise ValueError("A and omega must be float64 matrices")
    m, n = (int(x) for x in A.shape)
    l = int(omega.shape[0])
    if int(omega.shape[1]) != n:
        raise ValueError("omega must have n columns")
    A = A.contiguous()
    omega = omega.contiguous()
    U = torch.empty((m, k), dtype=torch.float64, device=A.device)
    s = torch.empty(k, dtype=torch.float64, device=A.device)
    V = torch.empty((n, k), dtype=torch.float64, device=A.device)
    _bind_stream(A.device)
    _check(lib().lrc_rsvd(A.data_ptr(), m, n, omega.data_ptr(), l, int(power_iters), int(k), U.data_ptr(),
                          s.data_ptr(), V.data_ptr()))
    return U, s, V


def tt_rsvd(T, ranks, omegas, power_iters: int = 0):
    """Randomized TT-SVD of the float64 device tensor T at TT ranks
    `ranks` (d-1 values), omegas[l] holding the test vectors of step l as
    rows.  Returns (cores, sigmas): float64 cores (r_{l-1}, n_l, r_l) and
    the kept singular values of every step."""
    import torch
    _dev(T, *omegas)
    if T.dtype != torch.float64 or any(o.dtype != torch.float64 for o in omegas):
        raise ValueError("T and the test matrices must be float64")
    dims = [int(x) for x in T.shape]
    d = len(dims)
    rk = [1] + [int(r) for r in ranks] + [1]
    if len(rk) != d + 1 or len(omegas) != d - 1:
        raise ValueError("need d-1 ranks and d-1 test matrices")
    T = T.contiguous()
    oms = [o.contiguous() for o in omegas]
    cores = [torch.empty((rk[l], dims[l], rk[l + 1]), dtype=torch.float64, device=T.device) for l in range(d)]
    sig = torch.empty(sum(rk[1:d]), dtype=torch.float64, device=T.device)
    D = (_i64 * d)(*dims)
    R = (_i64 * (d + 1))(*rk)
    S = (_i64 * (d - 1))(*[int(o.shape[0]) for o in oms])
    O = (_vp * (d - 1))(*[o.data_ptr() for o in oms])
    C = (_vp * d)(*[c.data_ptr() for c in cores])
    _bind_stream(T.device)
    _check(lib().lrc_tt_rsvd(T.data_ptr(), D, R, d, O, S, int(power_iters), C, sig.data_ptr()))
    sigmas, o = [], 0
    for r in rk[1:d]:
        sigmas.append(sig[o:o + r])
        o += r
    return cores, sigmas


def _result(res: CertResult) -> dict:
    out = {f: getattr(res, f) for f, _ in CertResult._fields_}
    for f in ("certified", "acc_nonincrease", "acc_win", "mem_win", "practical_win"):
        out[f] = bool(out[f])
    return out


def certify_matrix(sigma, U, s, V, Uh, sh, Vh, k: int, A=None) -> dict:
    """Matrix certificate for base rank k (FP64) vs rank k+1 stored as
    (Uh, sh, Vh).  sigma: host sequence of all min(m, n) singular values;
    U (m x k+1), s (k+1), V (n x k+1) float64; Uh, sh, Vh the same shapes
    in float32 or float16; A (m x n, float64) or None."""
    import numpy as np
    import torch
    sig = np.ascontiguousarray(np.asarray(sigma, dtype=np.float64))
    _need(U.dim() == 2 and V.dim() == 2, "U and V must be matrices")
    m, n, r = int(U.shape[0]), int(V.shape[0]), int(k) + 1
    _need(int(k) >= 1 and tuple(U.shape) == (m, r) and tuple(V.shape) == (n, r) and tuple(s.shape) == (r,),
          f"FP64 factors must have k + 1 = {r} columns: U {tuple(U.shape)}, s {tuple(s.shape)}, V {tuple(V.shape)}")
    for name, t in (("U", U), ("s", s), ("V", V)):
        if t.dtype != torch.float64:
            raise TypeError(f"{name} must be float64")
    for name, t, ref in (("Uh", Uh, U), ("sh", sh, s), ("Vh", Vh, V)):
        _need(tuple(t.shape) == tuple(ref.shape), f"{name} has shape {tuple(t.shape)}, want {tuple(ref.shape)}")
        if t.dtype != Uh.dtype or t.dtype not in (torch.float16, torch.float32, torch.float64):
            raise TypeError("Uh, sh, Vh must share one storage dtype")
    _need(sig.ndim == 1 and sig.size == min(m, n), f"sigma must hold all min(m, n) = {min(m, n)} singular values")
    if A is not None:
        _need(tuple(A.shape) == (m, n), f"A has shape {tuple(A.shape)}, want {(m, n)}")
        if A.dtype != torch.float64:
            raise TypeError("A must be float64")
    _dev(U, s, V, Uh, sh, Vh)
    if A is not None:
        _dev(A)
    a = CertArgs()
    a.kind = CERT_MATRIX
    a.prec = _prec_of(Uh)
    a.m, a.n, a.k = m, n, int(k)
    a.sigma = sig.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    a.n_sigma = len(sig)
    a.U, a.s, a.V = U.data_ptr(), s.data_ptr(), V.data_ptr()
    a.Uh, a.sh, a.Vh = Uh.data_ptr(), sh.data_ptr(), Vh.data_ptr()
    a.A = A.data_ptr() if A is not None else None
    res = CertResult()
    _bind_stream(U.device)
    _check(lib().lrc_certify(ctypes.byref(a), ctypes.byref(res)))
    return _result(res)


def certify_tt(T, base_cores, aug_cores, aug_cores_h) -> dict:
    """TT certificate: T dense FP64 of the trains' shape; FP64 base and
    augmented cores; the augmented cores as stored (FP32 or FP16), of the
    augmented cores' shapes."""
    import torch
    d = len(base_cores)
    _need(len(aug_cores) == d and len(aug_cores_h) == d, "the three trains must have the same number of cores")
    for cs in (base_cores, aug_cores, aug_cores_h):
        _check_train(cs)
    for cs in (base_cores, aug_cores):
        if cs[0].dtype != torch.float64:
            raise TypeError("base and augmented cores must be float64")
    dims, rb = tt_shape(base_cores)
    dims_a, ra = tt_shape(aug_cores)
    _need(dims_a == dims, f"augmented train has dims {dims_a}, base {dims}")
    for l in range(d):
        _need(tuple(aug_cores_h[l].shape) == tuple(aug_cores[l].shape),
              f"stored core {l} has shape {tuple(aug_cores_h[l].shape)}, want {tuple(aug_cores[l].shape)}")
    _need(T.numel() == math.prod(dims), f"T has {T.numel()} entries, want {math.prod(dims)}")
    if T.dtype != torch.float64:
        raise TypeError("T must be float64")
    _dev(T, *base_cores, *aug_cores, *aug_cores_h)
    a = CertArgs()
    a.kind = CERT_TT
    a.prec = _prec_of(aug_cores_h[0])
    a.d = d
    D = (_i64 * d)(*dims)
    RB = (_i64 * (d + 1))(*rb)
    RA = (_i64 * (d + 1))(*ra)
    PB = (_vp * d)(*[c.data_ptr() for c in base_cores])
    PA = (_vp * d)(*[c.data_ptr() for c in aug_cores])
    PH = (_vp * d)(*[c.data_ptr() for c in aug_cores_h])
    a.dims, a.ranks_base, a.ranks_aug = D, RB, RA
    a.cores_base, a.cores_aug, a.cores_aug_h = PB, PA, PH
    a.T = T.data_ptr()
    res = CertResult()
    _bind_stream(T.device)
    _check(lib().lrc_certify(ctypes.byref(a), ctypes.byref(res)))
    return _result(res)


def profile_enable(on: bool = True):
    _check(lib().lrc_profile_enable(1 if on else 0))


def profile_filter(label=None):
    """Time only launches labelled `label` (None: every launch)."""
    _check(lib().lrc_profile_filter(label.encode() if label else None))


def profile_reset():
    lib().lrc_profile_reset()


def mfma_ceiling(prec: str) -> float:
    """Measured matrix-core ceiling (TFLOP/s) of the kernels' MFMA
    instruction for prec ('fp64', 'fp32' or 'fp16') on the current device."""
    codes = {"fp64": 0, "fp32": 1, "fp16": 2}
    if prec not in codes:
        raise ValueError(f"prec must be one of {sorted(codes)}")
    out = ctypes.c_double()
    _check(lib().lrc_mfma_ceiling(codes[prec], ctypes.byref(out)))
    return float(out.value)


def profile_read() -> dict:
    """{kernel label: (launches, total milliseconds)} for every label seen."""
    L = lib()
    n = _check(L.lrc_profile_labels(None, 0))
    buf = ctypes.create_string_buffer(n + 1)
    L.lrc_profile_labels(buf, n + 1)
    out = {}
    for lab in filter(None, buf.value.decode().split(",")):
        cnt, ms = _i64(), ctypes.c_double()
        _check(L.lrc_profile_read(lab.encode(), ctypes.byref(cnt), ctypes.byref(ms)))
        out[lab] = (cnt.value, ms.value)
    return out


def shutdown():
    lib().lrc_shutdown()

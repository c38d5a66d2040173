"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/lrc.h declares, computes storage counts exactly, and
rejects bad arguments before touching the device."""
import ctypes

import numpy as np
import pytest

import oracle as O
from paper_2607_12969_amd import lrc

L = None


def setup_module():
    global L
    L = lrc.lib()


def test_exports_every_declared_symbol():
    declared = lrc.header_symbols()
    assert len(declared) >= 11
    for name in declared:
        assert hasattr(L, name), name
    assert L.lrc_version() == 1


@pytest.mark.parametrize("m,n,k", [(512, 256, 20), (8192, 8192, 257), (65536, 4096, 513), (1, 1, 1)])
def test_storage_bytes_match_oracle(m, n, k):
    for prec in ("fp64", "fp32", "fp16"):
        assert lrc.storage_bytes(m, n, k, prec) == O.storage_bytes(m, n, k, prec)


def test_tt_storage_bytes_match_oracle():
    cases = [((145, 145, 200), (1, 32, 32, 1)), ((16,) * 6, (1, 9, 17, 25, 17, 9, 1)), ((7,), (1, 1))]
    for dims, ranks in cases:
        for prec in ("fp64", "fp32", "fp16"):
            assert lrc.tt_storage_bytes(dims, ranks, prec) == O.tt_storage_bytes(dims, ranks, prec)


def test_storage_overflow_and_invalid():
    assert L.lrc_storage_bytes(2 ** 62, 2 ** 62, 10, 0) == -2
    assert L.lrc_storage_bytes(10, 10, 3, 7) == -1
    with pytest.raises(lrc.LrcError):
        lrc.tt_storage_bytes((4, 5), (2, 3, 1), "fp64")      # ranks[0] != 1


def test_apply_path_dispatch():
    assert lrc.apply_path(8192, 8192, 257, 1, "fp16") == lrc.PATH_STREAM
    assert lrc.apply_path(8192, 8192, 257, 8, "fp64") == lrc.PATH_STREAM
    assert lrc.apply_path(8192, 8192, 257, 9, "fp32") == lrc.PATH_MFMA
    assert lrc.apply_path(8192, 8192, 257, 4096, "fp16") == lrc.PATH_MFMA
    assert L.lrc_matrix_apply_path(10, 10, 11, 4, 0) == -1   # k > min(m, n)
    # the streaming path keeps T' (k x batch, accumulation type) in 64 KB of LDS
    assert lrc.apply_path(9000, 9000, 8192, 1, "fp64") == lrc.PATH_STREAM
    assert lrc.apply_path(9000, 9000, 8193, 1, "fp64") == lrc.PATH_MFMA
    assert lrc.apply_path(9000, 9000, 2048, 8, "fp32") == lrc.PATH_STREAM
    assert lrc.apply_path(9000, 9000, 2049, 8, "fp32") == lrc.PATH_MFMA
    assert L.lrc_set_apply_path(3) == -1
    assert L.lrc_set_apply_path(0) == 0


def _apply(ptrs, m, n, k, b, prec):
    return L.lrc_matrix_apply(*ptrs, m, n, k, b, prec)


def test_apply_argument_errors():
    good = [0x10000, 0x20000, 0x30000, 0x40000, 0x90000000]
    assert _apply([0] + good[1:], 10, 10, 3, 4, 0) == -1                 # NULL
    assert _apply(good, 0, 10, 3, 4, 0) == -1                           # m < 1
    assert _apply(good, 10, 10, 0, 4, 0) == -1                          # k < 1
    assert _apply(good, 10, 10, 11, 4, 0) == -1                         # k > min(m, n)
    assert _apply(good, 10, 10, 3, 0, 0) == -1                          # batch < 1
    assert _apply(good, 10, 10, 3, 4, 5) == -1                          # bad precision
    assert _apply(good, 2 ** 40, 2 ** 40, 3, 2 ** 40, 0) == -2          # overflow
    overl = [0x10000, 0x20000, 0x30000, 0x40000, 0x10008]               # Y overlaps U
    assert _apply(overl, 10, 10, 3, 4, 0) == -1
    assert b"overlaps" in L.lrc_last_error()


def test_noalloc_apply_checks_on_the_host():
    """The allocation-free apply validates like lrc_matrix_apply and rejects
    sizes whose plan needs more than its fixed scratch before any device
    call (T' alone of a 65536 x 4096 FP64 apply at rank 512 and batch 20000
    is 82 MB)."""
    good = [0x10000, 0x20000, 0x30000, 0x40000, 0x90000000]
    f = L.lrc_matrix_apply_noalloc
    assert f(0, *good[1:], 10, 10, 3, 4, 0) == -1                          # NULL
    assert f(*good, 10, 10, 11, 4, 0) == -1                                # k > min(m, n)
    assert f(*good, 65536, 4096, 512, 20000, 0) == -1
    assert b"scratch" in L.lrc_last_error()


def _tt(dims, ranks, d, prec=0, cores=None, out=0x90000000):
    D = (ctypes.c_int64 * max(1, len(dims)))(*dims)
    R = (ctypes.c_int64 * max(1, len(ranks)))(*ranks)
    if cores is None:
        cores = [0x10000 * (i + 1) for i in range(max(1, d))]
    P = (ctypes.c_void_p * len(cores))(*cores)
    return L.lrc_tt_reconstruct(P, D, R, d, out, prec)


def test_tt_argument_errors():
    assert _tt((4, 5), (1, 3, 1), 0) == -1                  # d < 1
    assert _tt((4, 5), (1, 3, 1), 17) == -1                 # d > max
    assert _tt((4, 5), (2, 3, 1), 2) == -1                  # ranks[0] != 1
    assert _tt((4, 5), (1, 3, 2), 2) == -1                  # ranks[d] != 1
    assert _tt((4, 0), (1, 3, 1), 2) == -1                  # dim < 1
    assert _tt((4, 5), (1, 0, 1), 2) == -1                  # rank < 1
    assert _tt((4, 5), (1, 513, 1), 2) == -1                # rank above the limit
    assert _tt((4, 5), (1, 3, 1), 2, prec=9) == -1          # bad precision
    assert _tt((4, 5), (1, 3, 1), 2, cores=[0x10000, 0]) == -1
    assert _tt((2 ** 40, 2 ** 40), (1, 3, 1), 2) == -2      # entry count overflow
    assert _tt((4, 5), (1, 3, 1), 2, out=0x10008) == -1     # output overlaps a core


def test_certify_argument_errors():
    a = lrc.CertArgs()
    r = lrc.CertResult()
    a.kind = 5
    a.prec = 1
    assert L.lrc_certify(ctypes.byref(a), ctypes.byref(r)) == -1
    a.kind = lrc.CERT_MATRIX
    a.m, a.n, a.k = 10, 8, 8                                 # k + 1 > min(m, n)
    sig = np.linspace(1, 0.1, 8)
    a.sigma = sig.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    a.n_sigma = 8
    assert L.lrc_certify(ctypes.byref(a), ctypes.byref(r)) == -1
    a.k = 3
    a.U = a.s = a.V = a.Uh = a.sh = a.Vh = 0x10000
    bad = np.array([1.0, 2.0, 0.5, 0.1, 0.05, 0.04, 0.03, 0.02])   # not non-increasing
    a.sigma = bad.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    a.n_sigma = 8
    assert L.lrc_certify(ctypes.byref(a), ctypes.byref(r)) == -1
    assert b"non-increasing" in L.lrc_last_error()
    a.kind = lrc.CERT_TT
    a.d = 0
    assert L.lrc_certify(ctypes.byref(a), ctypes.byref(r)) == -1


def test_certify_rejects_truncated_spectrum():
    """The tails E_k, E_{k+1} of Thm thm:matrix_rank_compensation sum over
    the whole spectrum: a spectrum cut after sigma_{k+1} (say, from a rank-k
    factorization) would make E_{k+1} = 0 and certify on eta <= sigma_{k+1}
    alone, so anything but min(m, n) values is rejected before any device
    call."""
    a = lrc.CertArgs()
    r = lrc.CertResult()
    a.kind = lrc.CERT_MATRIX
    a.prec = lrc.FP16
    a.m, a.n, a.k = 10, 8, 3
    a.U = a.s = a.V = a.Uh = a.sh = a.Vh = 0x10000
    sig = np.linspace(1.0, 0.1, 8)
    a.sigma = sig.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    for n_sigma in (4, 7, 9):                                 # k + 1, one short, one too many
        a.n_sigma = n_sigma
        assert L.lrc_certify(ctypes.byref(a), ctypes.byref(r)) == -1
        assert b"min(m, n)" in L.lrc_last_error()


def test_valid_call_without_gpu_reports_no_device():
    try:
        import torch
        if torch.cuda.is_available():
            pytest.skip("a GPU is present")
    except ImportError:
        pass
    good = [0x10000, 0x20000, 0x30000, 0x40000, 0x90000000]
    assert _apply(good, 10, 10, 3, 4, 0) == -5


def test_round_argument_errors():
    n = ctypes.c_int64(0)
    assert L.lrc_round(None, 0x20000, 8, 1, None) == -1                  # NULL x
    assert L.lrc_round(0x10000, None, 8, 1, None) == -1                  # NULL y
    assert L.lrc_round(0x10000, 0x20000, -1, 1, None) == -1              # count < 0
    assert L.lrc_round(0x10000, 0x20000, 8, 7, None) == -1               # bad precision
    assert L.lrc_round(0x10000, 0x10010, 8, 2, ctypes.byref(n)) == -1    # y overlaps x
    assert L.lrc_round(0x10000, 0x20000, 2 ** 61, 2, None) == -2         # byte count overflow


def _gauge(dims, ranks, d, cores=None):
    D = (ctypes.c_int64 * max(1, len(dims)))(*dims)
    R = (ctypes.c_int64 * max(1, len(ranks)))(*ranks)
    if cores is None:
        cores = [0x1000000 * (i + 1) for i in range(max(1, d))]
    P = (ctypes.c_void_p * len(cores))(*cores)
    return L.lrc_tt_left_orthogonalize(P, D, R, d)


def test_gauge_argument_errors():
    assert _gauge((4, 5), (1, 3, 1), 0) == -1                 # d < 1
    assert _gauge((4, 5), (2, 3, 1), 2) == -1                 # ranks[0] != 1
    assert _gauge((4, 5), (1, 3, 1), 2, cores=[0x1000000, 0]) == -1
    assert _gauge((200, 200), (1, 97, 1), 2) == -1            # rank above the gauge's limit
    assert _gauge((4, 3, 60), (1, 3, 13, 1), 3) == -1         # core 1: 3 * 3 = 9 rows < 13 columns
    assert b"rows" in L.lrc_last_error()
    assert _gauge((4, 5), (1, 3, 1), 2, cores=[0x1000000, 0x1000008]) == -1   # cores overlap
    assert b"overlaps" in L.lrc_last_error()
    assert _gauge((2 ** 40, 2 ** 40), (1, 3, 1), 2) == -2     # entry count overflow


def test_memory_matched_rank_matches_oracle():
    """Pure host function: equal to the oracle's search (integers, exact),
    including the paper's (17, 17) at its four budgets."""
    cases = [((145, 145, 200), 36), ((610, 340, 103), 36), ((83, 86, 204), 36), ((512, 217, 204), 36),
             ((4, 5, 6), 3), ((16,) * 6, 12), ((128, 24, 64, 64), 20), ((3, 3), 5)]
    for dims, Rc in cases:
        for prec in ("fp16", "fp32"):
            budget = O.tt_storage_bytes(dims, O.capped_ranks(dims, Rc), prec)
            for b in (budget, budget - 1, budget + 1, 8, 10 ** 12):
                assert lrc.memory_matched_rank(dims, b) == O.memory_matched_rank(dims, b), (dims, b)


def test_quality_argument_errors():
    q = lrc.Quality()
    assert L.lrc_band_quality(None, 0x10000, 4, 4, 0, 1.0, ctypes.byref(q)) == -1
    assert L.lrc_band_quality(0x10000, 0x20000, 0, 4, 0, 1.0, ctypes.byref(q)) == -1
    assert L.lrc_band_quality(0x10000, 0x20000, 4, 4, 9, 1.0, ctypes.byref(q)) == -1
    assert L.lrc_band_quality(0x10000, 0x20000, 2 ** 40, 2 ** 40, 0, 1.0, ctypes.byref(q)) == -2
    D = (ctypes.c_int64 * 1)(5)
    R = (ctypes.c_int64 * 2)(1, 1)
    P = (ctypes.c_void_p * 1)(0x10000)
    assert L.lrc_tt_quality(P, D, R, 1, 0, 0x20000, 1.0, ctypes.byref(q)) == -1     # d < 2
    out = (ctypes.c_int64 * 2)()
    assert L.lrc_tt_memory_matched_rank(D, 0, 100, out) == -1


def _rsvd(m, n, l, k, q=0, A=0x100000, Om=0x8000000, U=0x10000000, s=0x20000000, V=0x30000000):
    return L.lrc_rsvd(A, m, n, Om, l, q, k, U, s, V)


def test_rsvd_argument_errors():
    """Checked on the host before any device call (no GPU here)."""
    assert _rsvd(100, 80, 10, 5, A=0) == -1                    # NULL input
    assert _rsvd(0, 80, 10, 5) == -1                           # empty matrix
    assert _rsvd(100, 80, 10, 11) == -1                        # k > l
    assert _rsvd(100, 80, 10, 0) == -1                         # k < 1
    assert _rsvd(100, 80, 97, 5) == -1                         # above LRC_RSVD_MAX_SAMPLES
    assert _rsvd(100, 8, 10, 5) == -1                          # l > n
    assert b"exceed" in L.lrc_last_error()
    assert _rsvd(100, 80, 10, 5, q=9) == -1                    # too many power iterations
    assert _rsvd(100, 80, 10, 5, U=0x100000 + 8) == -1         # U overlaps A
    assert b"overlaps" in L.lrc_last_error()
    assert _rsvd(100, 80, 10, 5, V=0x10000000 + 16) == -1      # V overlaps U
    assert _rsvd(2 ** 40, 2 ** 40, 10, 5) == -2                # size overflow


def test_tt_rsvd_argument_errors():
    def call(dims, ranks, samples, omegas=None, cores=None, T=0x100000, q=0):
        d = len(dims)
        D = (ctypes.c_int64 * d)(*dims)
        R = (ctypes.c_int64 * (d + 1))(*ranks)
        S = (ctypes.c_int64 * max(d - 1, 1))(*samples)
        om = omegas or [0x4000000 * (l + 1) for l in range(d - 1)]
        co = cores or [0x40000000 + 0x4000000 * l for l in range(d)]
        O_ = (ctypes.c_void_p * max(d - 1, 1))(*om)
        C_ = (ctypes.c_void_p * d)(*co)
        return L.lrc_tt_rsvd(T, D, R, d, O_, S, q, C_, None)
    assert call((8, 9, 10), (1, 4, 5, 1), (6, 7), T=0) == -1
    assert call((8,), (1, 1), ()) == -1                           # d < 2
    assert call((8, 9, 10), (1, 4, 5, 1), (3, 7)) == -1           # rank 4 > 3 test vectors
    assert call((8, 9, 10), (1, 4, 5, 1), (6, 11)) == -1          # 11 test vectors > 10 columns of step 1
    assert b"step 1" in L.lrc_last_error()
    assert call((8, 9, 10), (1, 4, 5, 1), (6, 7), q=-1) == -1
    assert call((8, 9, 10), (1, 4, 5, 1), (6, 7), omegas=[0x4000000, 0]) == -1
    assert call((8, 9, 10), (1, 4, 5, 1), (6, 7), cores=[0x40000000, 0x40000000 + 64, 0x48000000]) == -1
    assert b"overlap" in L.lrc_last_error()
    assert call((8, 9, 10), (1, 4, 5, 1), (6, 7), cores=[0x100000 + 8, 0x44000000, 0x48000000]) == -1

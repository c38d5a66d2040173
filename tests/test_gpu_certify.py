"""GPU parity of the device-side certificate (Thm thm:matrix_rank_compensation,
Thm thm:tt_conditional, Algorithm alg:tt_compensation) against the oracle.

Verdicts, outcome codes and byte counts must be identical.  The Frobenius
quantities are FP64 reductions in a different order (and, for eta of the
matrix certificate, through the Gram matrices of the exact rounding
differences instead of a dense difference), so they are compared with
tolerances derived from FP64 rounding: the oracle's dense eta carries a
relative error of about eps ||A|| / eta (<= 1e-7 for FP32 storage)."""
import numpy as np
import pytest

import oracle as O
from paper_2607_12969_amd import synth
from conftest import read_golden
from parity import to_dev

pytestmark = pytest.mark.gpu

FLAGS = ("certified", "acc_nonincrease", "acc_win", "mem_win", "practical_win", "outcome",
         "bytes_base", "bytes_aug")


@pytest.fixture(scope="module")
def lrc():
    import torch
    from paper_2607_12969_amd import lrc as mod
    assert torch.cuda.is_available()
    mod.lib()
    return mod


def _stored(a, prec):
    return np.ascontiguousarray(a).astype({"fp64": np.float64, "fp32": np.float32, "fp16": np.float16}[prec])


def _matrix(lrc, sigma, U, s, V, k, prec, A=None):
    f64 = [np.ascontiguousarray(x) for x in (U, s, V)]
    got = lrc.certify_matrix(sigma, *[to_dev(x) for x in f64], *[to_dev(_stored(x, prec)) for x in f64], k,
                             A=to_dev(A) if A is not None else None)
    want = O.matrix_certificate(sigma, *f64, k, prec, A=A)
    return got, want


def _compare(got, want, eta_rtol, err_rtol=1e-9, e_atol=0.0, check_flags=True):
    for f in ("E_base", "E_aug", "norm_ref"):
        assert abs(got[f] - want[f]) <= 1e-12 * abs(want[f]) + e_atol, f
    if want["eta"] == 0.0:
        assert got["eta"] <= 1e-15 * want["norm_ref"]
    else:
        assert abs(got["eta"] - want["eta"]) <= eta_rtol * want["eta"], (got["eta"], want["eta"])
    if not np.isnan(want["err_new"]):
        assert abs(got["err_new"] - want["err_new"]) <= err_rtol * want["err_new"] + e_atol
    if check_flags:
        for f in FLAGS:
            assert got[f] == want[f], (f, got[f], want[f])


@pytest.mark.parametrize("prec", ["fp64", "fp32", "fp16"])
def test_matrix_small_with_dense(lrc, prec):
    w = synth.matrix_small()
    U, S, Vt = O.svd(w["A"])
    k = w["k"]
    print(f"certify 512x256 prec={prec}", flush=True)
    got, want = _matrix(lrc, S, U[:, :k + 1], S[:k + 1], Vt[:k + 1].T, k, prec, A=w["A"])
    _compare(got, want, eta_rtol=1e-6)


def test_matrix_failing_case(lrc):
    m, n, k = 300, 200, 30
    rng = synth.rng_for(synth.W_RANDOM, 40)
    U = synth.haar(rng, m, n)
    V = synth.haar(rng, n, n)
    sig = np.concatenate([np.ones(k), 1e-6 * 0.5 ** np.arange(n - k)])
    A = O.lowrank_dense(U, sig, V)
    for prec in ("fp32", "fp16"):
        got, want = _matrix(lrc, sig, U[:, :k + 1], sig[:k + 1], V[:, :k + 1], k, prec, A=A)
        _compare(got, want, eta_rtol=1e-6, err_rtol=1e-6)
    assert not got["certified"] and got["outcome"] == 0


_CACHE = {}


def _square():
    # one 8192 x 8192 matrix for every k (its leading 257 singular triplets)
    if "sq" not in _CACHE:
        _CACHE["sq"] = synth.matrix_square(kmax=256, batch=1)
    return _CACHE["sq"]


def _tail():
    if "tail" not in _CACHE:
        _CACHE["tail"] = synth.matrix_tail(kmax=512, batch=1)
    return _CACHE["tail"]


@pytest.mark.parametrize("k", [64, 128, 256])
@pytest.mark.parametrize("prec", ["fp32", "fp16"])
def test_matrix_square_workload(lrc, k, prec):
    w = _square()
    print(f"certify 8192^2 k={k} prec={prec}", flush=True)
    got, want = _matrix(lrc, w["sigma"], w["U"][:, :k + 1], w["sigma"][:k + 1], w["V"][:, :k + 1], k, prec)
    _compare(got, want, eta_rtol=1e-6)
    assert abs(want["margin"]) > 1e-6 * want["E_base"]   # verdict not at the boundary


@pytest.mark.parametrize("k", [64, 256, 512])
@pytest.mark.parametrize("prec", ["fp32", "fp16"])
def test_matrix_tail_workload(lrc, k, prec):
    w = _tail()
    print(f"certify 65536x4096 k={k} prec={prec}", flush=True)
    got, want = _matrix(lrc, w["sigma"], w["U"][:, :k + 1], w["sigma"][:k + 1], w["V"][:, :k + 1], k, prec)
    _compare(got, want, eta_rtol=1e-6)
    assert abs(want["margin"]) > 1e-6 * want["E_base"]


@pytest.fixture(scope="module")
def square_dense():
    """The 8192 x 8192 workload formed densely (full Haar singular vectors),
    so that err_new = ||A - A_hat_{k+1}||_F is measured against A itself."""
    return synth.matrix_square_dense(kmax=256)


@pytest.mark.parametrize("k", [64, 256])
@pytest.mark.parametrize("prec", ["fp32", "fp16"])
def test_matrix_square_err_new(lrc, square_dense, k, prec):
    """err_new at the 8192 x 8192 size: the dense FP64 matrix-core pass over
    A (512 MB) against the oracle's dense difference, plus the accuracy-win
    flags it decides (Sec. 4.1 vocabulary)."""
    w = square_dense
    print(f"certify 8192^2 with A k={k} prec={prec}", flush=True)
    got, want = _matrix(lrc, w["sigma"], w["U"][:, :k + 1], w["sigma"][:k + 1], w["V"][:, :k + 1], k, prec,
                        A=w["A"])
    _compare(got, want, eta_rtol=1e-6, err_rtol=1e-9)
    # E_k^2 = E_{k+1}^2 + sigma_{k+1}^2 and err_new^2 = E_{k+1}^2 + eta^2 up to the
    # cross term, so err_new sits within eta of E_{k+1}
    assert abs(got["err_new"] - got["E_aug"]) <= got["eta"] * (1 + 1e-6) + 1e-12 * got["norm_ref"]


@pytest.mark.parametrize("prec", ["fp32", "fp16"])
def test_matrix_eta_exact_on_device(lrc, prec):
    """The device eta (Gram matrices of the exact rounding differences) on a
    factorization whose only rounding is in s, with every rounding error
    known: eta = h sqrt(3311) in closed form (see the oracle pin)."""
    from test_oracle_certificate import exact_eta_case
    U, s, V, sigma, exact = exact_eta_case(prec)
    got, want = _matrix(lrc, sigma, U, s, V, 20, prec)
    assert abs(got["eta"] - exact) <= 1e-14 * exact, (got["eta"], exact)
    assert abs(want["eta"] - exact) <= 2.0 ** -52 * exact
    for f in FLAGS:
        assert got[f] == want[f], f


def _tt(lrc, T, base, aug, prec):
    got = lrc.certify_tt(to_dev(T), [to_dev(c) for c in base], [to_dev(c) for c in aug],
                         [to_dev(_stored(c, prec)) for c in aug])
    want = O.tt_certificate(T, base, aug, prec)
    return got, want


@pytest.mark.parametrize("table", ["tt_three_way_detail.csv", "tt_six_way_detail.csv"])
def test_tt_paper_tables_on_device(lrc, table):
    """The device certificate reproduces the printed digits of the paper's
    synthetic TT tables (Sec. 7.2 / 7.3) from the oracle's TT-SVD cores."""
    gens = {"decay_3d": synth.decay_3d, "hilbert_3d": synth.hilbert_3d,
            "hilbert_6d": synth.hilbert_6d, "decay_6d": synth.decay_6d}
    cache = {}
    for row in read_golden(table):
        name = row["dataset"]
        if name not in cache:
            cache[name] = (gens[name](), {})
        T, bases = cache[name]
        R, Rp, prec = int(row["R"]), int(row["Rplus"]), row["prec"]
        if R not in bases:
            bases[R] = O.tt_svd(T, ranks=[R] * (T.ndim - 1))
        aug = O.left_orthogonalize(O.tt_svd(T, ranks=[Rp] * (T.ndim - 1)))
        print(f"certify tt {name} {R}->{Rp} {prec}", flush=True)
        got, want = _tt(lrc, T, bases[R], aug, prec)
        nT = got["norm_ref"]
        assert f"{got['E_base'] / nT:.2e}" == row["E_R"]
        assert f"{got['err_new'] / nT:.2e}" == row["new_error"]
        assert f"{got['eta'] / nT:.2e}" == row["eta"]
        assert ("Yes" if got["certified"] else "No") == row["cert"]
        assert f"{got['bytes_aug'] / got['bytes_base']:.2f}" == row["mem_ratio"]
        _compare(got, want, eta_rtol=1e-6, err_rtol=1e-6, e_atol=1e-13 * nT)


def test_tt_cube_workload(lrc):
    """256^3 generator tensor: TT-SVD at tolerance 1e-4, ranks + 1."""
    T = O.tt_full(synth.tt_cube_cores())
    for prec in ("fp32", "fp16"):
        r = O.tt_compensation(T, eps=1e-4, delta=1, prec=prec)
        print(f"certify tt 256^3 {r['ranks_base']}->{r['ranks_aug']} {prec}", flush=True)
        got, want = _tt(lrc, T, r["base_cores"], r["aug_cores"], prec)
        _compare(got, want, eta_rtol=1e-6, err_rtol=1e-6, e_atol=1e-12 * want["norm_ref"])


def test_tt_sixway_workload(lrc):
    """16^6 with exact TT ranks (8,16,24,16,8): E_R is at round-off, so the
    verdict is 'No' for both precisions; E_R itself is only compared to the
    size of the FP64 rounding noise."""
    from test_gpu_tt import sixway_tensor
    T = sixway_tensor()
    base = O.tt_svd(T, ranks=[8, 16, 24, 16, 8])
    aug = O.left_orthogonalize(O.tt_svd(T, ranks=[9, 17, 25, 17, 9]))
    for prec in ("fp32", "fp16"):
        got, want = _tt(lrc, T, base, aug, prec)
        nT = want["norm_ref"]
        assert abs(got["E_base"] - want["E_base"]) <= 1e-13 * nT
        assert abs(got["eta"] - want["eta"]) <= 1e-6 * want["eta"]
        assert got["certified"] == want["certified"] == False   # noqa: E712
        assert got["outcome"] == want["outcome"] == 0


def _tt_labels(lrc, T, base, aug, prec):
    """Certificate plus the kernel labels its launches recorded."""
    lrc.profile_reset()
    lrc.profile_enable(True)
    try:
        got, want = _tt(lrc, T, base, aug, prec)
        labels = {k: v[0] for k, v in lrc.profile_read().items()}
    finally:
        lrc.profile_enable(False)
    return got, want, labels


@pytest.mark.parametrize("dims,rb,ra", [
    ((300, 200), (40,), (41,)),                 # d = 2: one middle and one last core
    ((12, 40, 30, 50), (10, 24, 20), (11, 25, 21)),
    # d = 3 by wave tiles, one case per register layout of the last product
    # (K extent 16, 32, 48, 64, 68), ragged n_1 and n_3
    ((37, 23, 45), (12, 13), (13, 14)),
    ((64, 7, 40), (20, 30), (21, 31)),
    ((48, 5, 100), (40, 44), (41, 45)),
    ((70, 3, 90), (62, 62), (63, 63)),
    ((80, 6, 70), (64, 64), (65, 65)),
    ((40, 8200, 5), (3, 4), (4, 5)),             # more tiles than resident waves
    ((100, 5, 90), (80, 80), (81, 81)),          # d = 3 beyond the wave layouts: LDS tiles
])
def test_tt_fused_certificate_shapes(lrc, dims, rb, ra):
    """The fused certificate kernel (one launch, no dense reconstructions)
    on two-, three- and four-core trains."""
    base = synth.random_tt_cores(dims, [1, *rb, 1], tag=21)
    aug = O.left_orthogonalize(synth.random_tt_cores(dims, [1, *ra, 1], tag=22))
    rng = np.random.default_rng(5)
    T = O.tt_full(base) + 1e-3 * rng.standard_normal(dims)
    for prec in ("fp32", "fp16"):
        got, want, labels = _tt_labels(lrc, T, base, aug, prec)
        assert labels.get("cert_tt_fused_f64") == 1 and "cert_sumsq5_f64" not in labels, labels
        _compare(got, want, eta_rtol=1e-6, err_rtol=1e-6, e_atol=1e-12 * want["norm_ref"])


def test_tt_certificate_split_kernels():
    """LRC_TT_CERT_SPLIT=1 (read once per process, so the cases run in a
    child process): the base train and the augmented pair as two wave-tile
    kernels; verdicts and sums as with the one-pass kernel."""
    import os
    import subprocess
    import sys
    script = os.path.join(os.path.dirname(os.path.abspath(__file__)), "cert_split_case.py")
    print("certify tt split kernels", flush=True)
    r = subprocess.run([sys.executable, "-u", script], env=dict(os.environ, LRC_TT_CERT_SPLIT="1"),
                       capture_output=True, text=True, timeout=110)
    print(r.stdout[-4000:], r.stderr[-2000:], flush=True)
    assert r.returncode == 0
    assert r.stdout.count(" ok") == 6


def test_tt_certificate_unfused_fallback(lrc):
    """Ranks whose three on-chip interface sets exceed the fused kernel's LDS
    budget take the dense path: three FP64 reconstructions and one pass of
    sums over the tensors."""
    dims = (256, 4, 256)
    base = synth.random_tt_cores(dims, [1, 200, 200, 1], tag=23)
    aug = O.left_orthogonalize(synth.random_tt_cores(dims, [1, 201, 201, 1], tag=24))
    rng = np.random.default_rng(6)
    T = O.tt_full(base) + 1e-3 * rng.standard_normal(dims)
    got, want, labels = _tt_labels(lrc, T, base, aug, "fp16")
    assert labels.get("cert_tt_fused_f64") == 3 and labels.get("cert_sumsq5_f64") == 1, labels
    _compare(got, want, eta_rtol=1e-6, err_rtol=1e-6, e_atol=1e-12 * want["norm_ref"])


@pytest.mark.parametrize("schedule", [(64, 65), (32, 33), (32, 36)])
@pytest.mark.parametrize("prec", ["fp32", "fp16"])
def test_tt_hyperspectral_workload(lrc, hyper, schedule, prec):
    """The benchmark's TT certificate input: the normalized 512 x 512 x 224
    cube with its own TT-SVD, FP64 base (64,64) or (32,32) against the
    compensated (65,65), (33,33) or (36,36) stored in FP32 / FP16.  Verdicts,
    outcome and bytes must equal the oracle's; the sums agree to FP64
    reduction-order rounding."""
    T, base, aug = hyper
    rb, ra = schedule
    print(f"certify tt 512x512x224 ({rb},{rb})->({ra},{ra}) {prec}", flush=True)
    got, want = _tt(lrc, T, base[rb], aug[ra], prec)
    print(f"  eta/|T| {want['eta'] / want['norm_ref']:.3e} E_R {want['E_base']:.6e} E_R+ {want['E_aug']:.6e} "
          f"certified {want['certified']}", flush=True)
    assert abs(want["margin"]) > 1e-9 * want["E_base"]      # verdict not at the boundary
    _compare(got, want, eta_rtol=1e-6, err_rtol=1e-6, e_atol=1e-12 * want["norm_ref"])


def test_tt_certificate_on_benchmark_cores(lrc, hyper):
    """The certificate verdicts the benchmark prints come from its own
    fixed-rank TT-SVD of the cube (LAPACK, for speed); the device certificate
    on exactly those cores must equal the oracle's on them."""
    import bench
    T = hyper[0]
    base = bench.tt_svd_fixed(T, (64, 64))
    aug = bench.tt_svd_fixed(T, (65, 65))
    for prec in ("fp32", "fp16"):
        print(f"certify tt benchmark cores (64,64)->(65,65) {prec}", flush=True)
        got, want = _tt(lrc, T, base, aug, prec)
        assert abs(want["margin"]) > 1e-9 * want["E_base"]
        _compare(got, want, eta_rtol=1e-6, err_rtol=1e-6, e_atol=1e-12 * want["norm_ref"])

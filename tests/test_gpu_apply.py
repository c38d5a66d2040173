"""GPU parity of the factor apply Y = U diag(s) V^T X (Sec. 4.4 eq.
gpu_matrix_apply) against the oracle on the same stored values.

Tolerances (relative Frobenius error vs the oracle's FP64 evaluation of the
stored factors): 1e-12 FP64, 1e-5 FP32, 2e-3 FP16 with FP32 accumulation.
Every output is compared, the 8192 x 8192 and 65536 x 4096 workloads
included; those also pass a per-tile Frobenius check and the componentwise
bound of Lemma lem:dot (Sec. 5.2) on every entry."""
import numpy as np
import pytest

import oracle as O
from paper_2607_12969_amd import synth
from parity import PRECS, TOL, apply_bound, componentwise_ratio, rel_fro, stored_pair, tile_rel_fro_max, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lrc():
    import torch
    from paper_2607_12969_amd import lrc as mod
    assert torch.cuda.is_available()
    mod.lib()
    yield mod
    mod.set_apply_path(mod.PATH_AUTO)


def _run(lrc, U, s, V, X, prec, path=0):
    import torch
    hs = [stored_pair(a, prec) for a in (U, s, V, X)]
    lrc.set_apply_path(path)
    try:
        Y = lrc.matrix_apply(*[to_dev(h) for h, _ in hs])
        torch.cuda.synchronize()
    finally:
        lrc.set_apply_path(0)
    return Y.cpu().numpy().astype(np.float64), [o for _, o in hs]


def _assert_parity(Y, u, s, v, x, prec):
    ref = O.apply(u, s, v, x)
    assert rel_fro(Y, ref) <= TOL[prec]
    assert componentwise_ratio(Y, ref, apply_bound(u, s, v, x, prec, ref)) <= 1.0


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("path", [1, 2])
def test_small_workload(lrc, prec, path):
    """512 x 256 matrix, base rank 20 (FP64) / compensated 21, batch 64
    (MFMA path) or the first 5 columns (streaming path)."""
    w = synth.matrix_small()
    U, S, Vt = O.svd(w["A"])
    k = 20 if prec == "fp64" else 21
    X = w["X"] if path == 2 else w["X"][:, :5]
    print(f"apply small prec={prec} path={path}", flush=True)
    Y, (u, s, v, x) = _run(lrc, U[:, :k], S[:k], Vt[:k].T, X, prec, path)
    _assert_parity(Y, u, s, v, x, prec)


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("m,n,k,b", [
    (1, 1, 1, 1), (37, 53, 5, 3), (53, 37, 37, 17), (300, 200, 129, 70),
    (1000, 700, 65, 129), (129, 4100, 100, 8), (64, 64, 64, 64), (2000, 3000, 33, 1),
])
def test_ragged_shapes_both_paths(lrc, prec, m, n, k, b):
    d = synth.random_factors(m, n, k, b, tag=m * 7 + n * 3 + k + b)
    for path in (0, 1, 2):
        if path == 1 and b > 8:
            continue
        print(f"apply ragged prec={prec} m={m} n={n} k={k} b={b} path={path}", flush=True)
        Y, (u, s, v, x) = _run(lrc, d["U"], d["s"], d["V"], d["X"], prec, path)
        _assert_parity(Y, u, s, v, x, prec)


@pytest.mark.parametrize("tile", ["64", "128"])
def test_forced_tile_edges(tile):
    """The matrix-core tiles pinned to 64 or 128 rows (LRC_APPLY_TILE, read
    once per process, so the cases run in a child process): shapes whose
    tiles are mostly edges, every precision, against the oracle."""
    import os
    import subprocess
    import sys
    script = os.path.join(os.path.dirname(os.path.abspath(__file__)), "forced_tile_case.py")
    print(f"apply forced tile {tile}", flush=True)
    r = subprocess.run([sys.executable, "-u", script], env=dict(os.environ, LRC_APPLY_TILE=tile),
                       capture_output=True, text=True, timeout=110)
    print(r.stdout[-4000:], r.stderr[-2000:], flush=True)
    assert r.returncode == 0
    assert r.stdout.count(" ok") == 18


def test_stream_and_mfma_paths_agree(lrc):
    d = synth.random_factors(800, 600, 41, 8, tag=3)
    for prec in PRECS:
        y1, _ = _run(lrc, d["U"], d["s"], d["V"], d["X"], prec, 1)
        y2, _ = _run(lrc, d["U"], d["s"], d["V"], d["X"], prec, 2)
        assert rel_fro(y1, y2) <= 2 * TOL[prec]


@pytest.mark.parametrize("b", [1, 8, 256])
def test_deterministic(lrc, b):
    """Bitwise equal results on repeated calls: the split sums are added in a
    fixed order whatever order the workgroups run in (for the streaming path,
    whichever workgroup finishes a column block last)."""
    d = synth.random_factors(3000, 9000, 65, b, tag=4)
    for prec in PRECS:
        y1, _ = _run(lrc, d["U"], d["s"], d["V"], d["X"], prec, 0)
        for _ in range(3):
            y2, _ = _run(lrc, d["U"], d["s"], d["V"], d["X"], prec, 0)
            assert np.array_equal(y1, y2), prec


def _full(lrc, U, s, V, X, prec, label):
    """Every output of the apply against the oracle on the same stored values:
    the relative Frobenius tolerance over the whole output and over every
    64 x 64 tile, and the componentwise bound of Lemma lem:dot on every
    entry."""
    import torch
    hs = [stored_pair(a, prec) for a in (U, s, V, X)]
    print(f"apply {label} prec={prec} shape={hs[0][0].shape[0]}x{hs[3][0].shape[1]} k={hs[0][0].shape[1]}",
          flush=True)
    Y = lrc.matrix_apply(*[to_dev(h) for h, _ in hs])
    torch.cuda.synchronize()
    got = Y.cpu().numpy().astype(np.float64)
    del Y
    u, s_, v, x = [o for _, o in hs]
    ref = O.apply(u, s_, v, x)
    err = rel_fro(got, ref)
    assert err <= TOL[prec], (label, prec, err)
    tile = tile_rel_fro_max(got, ref)
    assert tile <= TOL[prec], (label, prec, "worst 64 x 64 tile", tile)
    ratio = componentwise_ratio(got, ref, apply_bound(u, s_, v, x, prec, ref))
    assert ratio <= 1.0, (label, prec, "componentwise bound exceeded", ratio)
    return err


@pytest.fixture(scope="module")
def square():
    return synth.matrix_square(kmax=256, batch=4096)


@pytest.mark.parametrize("k", [64, 128, 256])
@pytest.mark.parametrize("b", [1, 64, 4096])
def test_square_workload_full(lrc, square, k, b):
    """8192 x 8192, sigma_j = j^-1.5 (+1e-8 noise): FP64 at rank k, FP32 and
    FP16 at rank k + 1, batches 1, 64 and 4096; every output compared."""
    X = square["X"][:, :b]
    for prec in PRECS:
        r = k if prec == "fp64" else k + 1
        _full(lrc, square["U"][:, :r], square["sigma"][:r], square["V"][:, :r], X, prec, "8192^2")


@pytest.fixture(scope="module")
def tail():
    return synth.matrix_tail(kmax=512, batch=4096)


@pytest.mark.parametrize("k", [64, 256, 512])
@pytest.mark.parametrize("prec", PRECS)
def test_tail_workload_full(lrc, tail, k, prec):
    """65536 x 4096, sigma_j = max(exp(-j/40), 1e-6), batch 4096: FP64 at
    rank k, FP32/FP16 at k + 1; every one of the 268M outputs compared."""
    w = tail
    r = k if prec == "fp64" else k + 1
    _full(lrc, w["U"][:, :r], w["sigma"][:r], w["V"][:, :r], w["X"], prec, "65536x4096")


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("shift", [1, 3])
@pytest.mark.parametrize("b", [37, 129])
def test_unaligned_operands(lrc, prec, shift, b):
    """Operands whose base address is not 16-byte aligned (views `shift`
    elements into a buffer), with odd rank and batch so that every row is
    misaligned too: at batch 37 phase 2 reads U in place (one column tile),
    at batch 129 the operands go through the padded copy; both match the
    oracle."""
    import torch
    m, n, k = 300, 500, 65
    d = synth.random_factors(m, n, k, b, tag=9 + shift + b)
    hs = [stored_pair(a, prec) for a in (d["U"], d["s"], d["V"], d["X"])]
    views = []
    for h, _ in hs:
        buf = torch.zeros(h.size + shift, dtype=torch.from_numpy(h).dtype, device="cuda")
        v = buf[shift:].view(h.shape)
        v.copy_(torch.from_numpy(np.ascontiguousarray(h)))
        views.append(v)
    lrc.set_apply_path(2)
    try:
        Y = lrc.matrix_apply(*views)
        torch.cuda.synchronize()
    finally:
        lrc.set_apply_path(0)
    u, s, v, x = [o for _, o in hs]
    _assert_parity(Y.cpu().numpy().astype(np.float64), u, s, v, x, prec)


@pytest.mark.parametrize("prec", PRECS)
@pytest.mark.parametrize("m,n,b", [(494, 494, 256), (494, 494, 8192), (640, 192, 2048), (96, 96, 8192),
                                   (1536, 1536, 2048)])
@pytest.mark.parametrize("inc", [0, 1])
def test_timing_grid_shapes(lrc, prec, m, n, b, inc):
    """Shapes of the paper's matrix timing grid (base rank 40, compensated
    rank 41, batches 256 / 2048 / 8192, unit-norm samples), same-rank
    controls included; every output compared."""
    k = 40 + inc
    d = synth.random_factors(m, n, k, b, tag=900 + m + b + inc)
    X = d["X"] / np.linalg.norm(d["X"], axis=0, keepdims=True)
    print(f"apply grid prec={prec} m={m} n={n} k={k} b={b}", flush=True)
    Y, (u, s, v, x) = _run(lrc, d["U"], d["s"], d["V"], X, prec)
    assert rel_fro(Y, O.apply(u, s, v, x)) <= TOL[prec]


def test_large_rank_small_batch(lrc):
    """A rank whose T' does not fit the streaming path's 64 KB of LDS at
    batch 1 (FP64, k = 8200) takes the matrix-core path and is applied
    correctly."""
    m, n, k = 8300, 8250, 8200
    rng = synth.rng_for(synth.W_RANDOM, 30, k)
    U = synth.gaussian(rng, (m, k)) / np.sqrt(m)
    V = synth.gaussian(rng, (n, k)) / np.sqrt(n)
    s = 0.999 ** np.arange(k)
    X = synth.gaussian(rng, (n, 1))
    print("apply 8300x8250 k=8200 b=1 fp64", flush=True)
    Y, (u, s, v, x) = _run(lrc, U, s, V, X, "fp64")
    _assert_parity(Y, u, s, v, x, "fp64")

"""Pins for the oracle's fixed-memory quality measures and the memory-
matched FP64 rank (Sec. sec:hyperspectral_application): special cases whose
values follow from the definitions by hand, brute-force loops on tiny
inputs, and the memory-matched ranks and budgets the paper prints."""
import math

import numpy as np
import pytest

import oracle as O


def _cube(shape, seed, positive=True):
    rng = np.random.default_rng([12969, 60, seed])
    X = rng.standard_normal(shape)
    return np.abs(X) + 0.5 if positive else X


def test_identity_is_perfect():
    X = _cube((6, 5, 7), 1)
    q = O.band_quality(X, X)
    assert q["rel_err"] == 0.0 and q["psnr"] == math.inf
    assert q["ssim"] == pytest.approx(1.0, abs=1e-15)
    assert q["sam"] <= 1e-7 and q["sam_pixels"] == 30


def test_constant_offset_closed_form():
    """Xh = X + c: MSE_b = c^2 and, since the offset leaves variances and
    the covariance equal to var(x), the structure factors cancel and the
    SSIM variant reduces to its luminance term."""
    X = _cube((8, 9, 4), 2)
    c = 0.125
    q = O.band_quality(X, X + c)
    Xm = X.reshape(-1, 4)
    L = Xm.max(axis=0) - Xm.min(axis=0)
    assert q["psnr"] == pytest.approx(np.mean(20 * np.log10(L / c)), rel=1e-12)
    mu = Xm.mean(axis=0)
    C1 = (0.01 * L) ** 2
    lum = (2 * mu * (mu + c) + C1) / (mu ** 2 + (mu + c) ** 2 + C1)
    assert q["ssim"] == pytest.approx(float(np.mean(lum)), rel=1e-12)
    assert q["rel_err"] == pytest.approx(c * math.sqrt(X.size) / np.linalg.norm(X), rel=1e-12)


def test_spectral_angles():
    # scaled spectra: zero angle; orthogonal: pi/2; 60 degrees by hand
    X = np.array([[[1.0, 0.0], [1.0, 0.0], [2.0, 2.0]]])
    Xh = np.array([[[3.0, 0.0], [0.0, 5.0], [1.0 + math.sqrt(3), 1.0 - math.sqrt(3)]]])
    q = O.band_quality(X, Xh)
    # third pixel: (2,2) vs (1+sqrt3, 1-sqrt3): cos = 4/(sqrt8 sqrt8) = 1/2
    assert q["sam_pixels"] == 3
    assert q["sam"] == pytest.approx((0.0 + math.pi / 2 + math.pi / 3) / 3, rel=1e-12)


def test_zero_pixels_are_left_out_of_sam():
    X = np.array([[[0.0, 0.0], [1.0, 1.0], [1.0, 2.0]]])
    Xh = np.array([[[1.0, 0.0], [1.0, -1.0], [0.0, 0.0]]])
    q = O.band_quality(X, Xh)
    assert q["sam_pixels"] == 1 and q["sam"] == pytest.approx(math.pi / 2, rel=1e-14)


def test_constant_band_range_rule():
    assert O.band_range(np.full(5, 0.25)) == 1.0
    assert O.band_range(np.full(5, -3.0)) == 3.0
    assert O.band_range(np.array([0.5, -1.5, 2.0])) == 3.5
    X = np.zeros((3, 3, 2)); X[..., 0] = 0.25; X[..., 1] = 4.0
    q = O.band_quality(X, X + 0.1)
    assert q["psnr"] == pytest.approx(np.mean([20 * math.log10(1.0 / 0.1), 20 * math.log10(4.0 / 0.1)]), rel=1e-12)


def test_brute_force_loops_tiny():
    X = _cube((3, 4, 5), 3, positive=False)
    Xh = X + 0.05 * _cube((3, 4, 5), 4, positive=False)
    q = O.band_quality(X, Xh)
    P, B = 12, 5
    xs = X.reshape(P, B).tolist(); ys = Xh.reshape(P, B).tolist()
    ps, ss = [], []
    for b in range(B):
        col = [xs[p][b] for p in range(P)]; coly = [ys[p][b] for p in range(P)]
        L = max(col) - min(col)
        mse = sum((col[p] - coly[p]) ** 2 for p in range(P)) / P
        ps.append(20 * math.log10(L / math.sqrt(mse)))
        mx = sum(col) / P; my = sum(coly) / P
        vx = sum((v - mx) ** 2 for v in col) / P; vy = sum((v - my) ** 2 for v in coly) / P
        cxy = sum((col[p] - mx) * (coly[p] - my) for p in range(P)) / P
        c1, c2 = (0.01 * L) ** 2, (0.03 * L) ** 2
        ss.append((2 * mx * my + c1) * (2 * cxy + c2) / ((mx * mx + my * my + c1) * (vx + vy + c2)))
    ang = []
    for p in range(P):
        dot = sum(xs[p][b] * ys[p][b] for b in range(B))
        nx = math.sqrt(sum(v * v for v in xs[p])); ny = math.sqrt(sum(v * v for v in ys[p]))
        ang.append(math.acos(max(-1.0, min(1.0, dot / (nx * ny)))))
    assert q["psnr"] == pytest.approx(sum(ps) / B, rel=1e-12)
    assert q["ssim"] == pytest.approx(sum(ss) / B, rel=1e-12)
    assert q["sam"] == pytest.approx(sum(ang) / P, rel=1e-12)


# The paper's fixed-memory budgets: each dataset's FP16 rank-compensated
# (36, 36) storage, rounded to 0.38 / 0.89 / 0.23 / 0.59 MiB, and the
# memory-matched FP64 rank (17, 17) for every one of them.
@pytest.mark.parametrize("name,dims,mib", [
    ("Indian Pines", (145, 145, 200), 0.38), ("PaviaU", (610, 340, 103), 0.89),
    ("Salinas-A", (83, 86, 204), 0.23), ("Salinas", (512, 217, 204), 0.59)])
def test_memory_matched_rank_of_the_paper(name, dims, mib):
    budget = O.tt_storage_bytes(dims, O.capped_ranks(dims, 36), "fp16")
    assert round(budget / 2 ** 20, 2) == mib
    R, ranks = O.memory_matched_rank(dims, budget)
    assert R == 17 and ranks == [1, 17, 17, 1]


def test_memory_matched_rank_edges():
    dims = (4, 5, 6)
    # every rank capped at (4, 6): storage stops growing, the search ends there
    full = O.tt_storage_bytes(dims, [1, 4, 6, 1], "fp64")
    R, ranks = O.memory_matched_rank(dims, 10 * full)
    assert ranks == [1, 4, 6, 1]
    assert O.memory_matched_rank(dims, 8) == (0, None)
    one = O.tt_storage_bytes(dims, [1, 1, 1, 1], "fp64")
    assert O.memory_matched_rank(dims, one) == (1, [1, 1, 1, 1])

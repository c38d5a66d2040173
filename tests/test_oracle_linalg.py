"""Pins for the oracle's apply, reconstruction and factorizations.

Apply (Sec. 4.4 eq. gpu_matrix_apply) and TT evaluation (Sec. 5.1; Sec. 7.5
eq. gpu_tt_reconstruction) are pinned by closed forms with exactly
representable values, by brute force on tiny inputs and by the library
matrix product on special cases.  The QR / Jacobi SVD / TT-SVD used for the
offline factorizations are pinned by the Eckart-Young identity on a matrix
with a prescribed spectrum, by orthogonality, by the library SVD's singular
values and by exact recovery of tensors of known TT rank."""
import itertools
import math

import numpy as np
import pytest

import oracle as O
from paper_2607_12969_amd import synth


# ----------------------------------------------------------------- apply ---

def test_apply_rank1_closed_form_exact():
    # Y = s u (v^T X) with small integers: every partial sum is an exact
    # integer, so the result must be exact.
    u = np.array([[1.0], [-2.0], [3.0]])
    v = np.array([[2.0], [1.0], [0.0], [-1.0]])
    s = np.array([3.0])
    X = np.arange(8.0).reshape(4, 2) - 3.0
    expect = 3.0 * u @ (v.T @ X)
    np.testing.assert_array_equal(O.apply(u, s, v, X), expect)


def test_apply_brute_force_tiny():
    rng = np.random.default_rng([12969, 98, 0])
    m, n, k, b = 3, 4, 2, 2
    U, s, V, X = (rng.standard_normal((m, k)), rng.standard_normal(k),
                  rng.standard_normal((n, k)), rng.standard_normal((n, b)))
    Y = O.apply(U, s, V, X)
    for i, c in itertools.product(range(m), range(b)):
        ref = 0.0
        for j in range(k):
            t = 0.0
            for l in range(n):
                t += V[l, j] * X[l, c]
            ref += U[i, j] * (s[j] * t)
        assert Y[i, c] == ref   # same order of operations: bitwise equal


@pytest.mark.parametrize("m,n,k,b", [(1, 1, 1, 1), (37, 19, 5, 3), (200, 130, 33, 70), (64, 256, 21, 1)])
def test_apply_matches_library_product(m, n, k, b):
    rng = np.random.default_rng([12969, 98, m, n, k, b])
    U, s, V, X = (rng.standard_normal((m, k)), rng.standard_normal(k),
                  rng.standard_normal((n, k)), rng.standard_normal((n, b)))
    Y = O.apply(U, s, V, X)
    ref = (U * s) @ (V.T @ X)
    assert np.linalg.norm(Y - ref) <= 1e-13 * np.linalg.norm(ref)
    # the transposed statement of the paper, Y_p = [(X_p V) diag(s)] U^T
    ref_p = ((X.T @ V) * s) @ U.T
    assert np.linalg.norm(Y - ref_p.T) <= 1e-13 * np.linalg.norm(ref)


def test_lowrank_dense_matches_library():
    rng = np.random.default_rng([12969, 98, 5])
    U, s, V = rng.standard_normal((40, 7)), rng.standard_normal(7), rng.standard_normal((30, 7))
    A = O.lowrank_dense(U, s, V)
    ref = (U * s) @ V.T
    assert np.linalg.norm(A - ref) <= 1e-14 * np.linalg.norm(ref)


# -------------------------------------------------------------------- TT ---

@pytest.mark.parametrize("dims,ranks", [
    ((5,), (1, 1)),
    ((3, 4), (1, 2, 1)),
    ((2, 3, 4), (1, 2, 3, 1)),
    ((3, 1, 4, 2, 5), (1, 3, 2, 4, 2, 1)),
    ((4, 4, 4, 4), (1, 4, 7, 4, 1)),
])
def test_tt_chain_equals_slice_product(dims, ranks):
    rng = np.random.default_rng([12969, 97, len(dims)])
    cores = [rng.standard_normal((ranks[l], dims[l], ranks[l + 1])) for l in range(len(dims))]
    full = O.tt_full(cores)
    assert full.shape == tuple(dims)
    for idx in itertools.product(*[range(n) for n in dims]):
        # brute force in Python, slice by slice
        v = cores[0][:, idx[0], :]
        for l in range(1, len(dims)):
            v = v @ cores[l][:, idx[l], :]
        ref = float(v[0, 0])
        assert abs(full[idx] - ref) <= 1e-14 * (1 + abs(ref))
        assert abs(O.tt_entry(cores, idx) - ref) <= 1e-14 * (1 + abs(ref))


def test_tt_two_cores_is_a_matrix_product():
    rng = np.random.default_rng([12969, 97, 11])
    G1 = rng.standard_normal((1, 30, 6))
    G2 = rng.standard_normal((6, 20, 1))
    ref = G1[0] @ G2[:, :, 0]
    full = O.tt_full([G1, G2])
    assert np.linalg.norm(full - ref) <= 1e-14 * np.linalg.norm(ref)


def test_tt_rank_one_is_an_outer_product():
    rng = np.random.default_rng([12969, 97, 12])
    vs = [rng.standard_normal(n) for n in (4, 5, 6)]
    cores = [v.reshape(1, -1, 1) for v in vs]
    ref = np.einsum("i,j,k->ijk", *vs)
    np.testing.assert_allclose(O.tt_full(cores), ref, rtol=1e-15, atol=0)


def test_tt_storage_counts():
    # sum_l R_{l-1} n_l R_l (Sec. 5.1) and the exact uniform 3-core ratio
    # (b/64)(R+delta)(R+delta+2)/(R(R+2)) of Sec. 6.1 for n_l = n
    assert O.tt_storage_count((10, 20, 30), (1, 3, 4, 1)) == 10 * 3 + 3 * 20 * 4 + 4 * 30
    for n, R, dl, prec, b in ((60, 4, 1, "fp16", 16), (100, 8, 4, "fp32", 32), (12, 16, 4, "fp16", 16)):
        base = O.tt_storage_bytes((n, n, n), (1, R, R, 1), "fp64")
        aug = O.tt_storage_bytes((n, n, n), (1, R + dl, R + dl, 1), prec)
        expect = (b / 64) * (R + dl) * (R + dl + 2) / (R * (R + 2))
        assert abs(aug / base - expect) < 1e-15


# ------------------------------------------------------- QR, SVD, TT-SVD ---

@pytest.mark.parametrize("m,n", [(1, 1), (7, 3), (50, 50), (300, 40)])
def test_qr_properties(m, n):
    rng = np.random.default_rng([12969, 96, m, n])
    A = rng.standard_normal((m, n))
    Q, R = O.qr(A)
    assert np.linalg.norm(Q @ R - A) <= 1e-13 * np.linalg.norm(A)
    assert np.linalg.norm(Q.T @ Q - np.eye(n)) <= 1e-13 * max(1, n)
    assert np.all(np.triu(R) == R) and np.all(np.diag(R) >= 0)
    # unique with diag(R) >= 0: equals the library R up to the row signs
    Rl = np.linalg.qr(A)[1]
    np.testing.assert_allclose(R, np.sign(np.diag(Rl))[:, None] * Rl, rtol=0,
                               atol=1e-12 * max(1.0, np.abs(Rl).max()))


@pytest.mark.parametrize("m,n,rank", [(40, 40, 40), (120, 30, 30), (30, 120, 30), (80, 60, 12), (5, 300, 5)])
def test_svd_against_library_values(m, n, rank):
    rng = np.random.default_rng([12969, 95, m, n])
    A = rng.standard_normal((m, rank)) @ rng.standard_normal((rank, n))
    U, S, Vt = O.svd(A)
    ref = np.linalg.svd(A, compute_uv=False)
    p = min(m, n)
    assert S.shape == (p,)
    assert np.all(np.diff(S) <= 0)
    np.testing.assert_allclose(S[:rank], ref[:rank], rtol=1e-12, atol=0)
    assert np.all(S[rank:] <= 1e-13 * S[0])
    assert np.linalg.norm((U * S) @ Vt - A) <= 1e-13 * np.linalg.norm(A)
    assert np.linalg.norm(U[:, :rank].T @ U[:, :rank] - np.eye(rank)) <= 1e-13 * p
    assert np.linalg.norm(Vt @ Vt.T - np.eye(p)) <= 1e-13 * p


def test_eckart_young_on_prescribed_spectrum():
    """The 512 x 256 workload has sigma_j = 10^(-4(j-1)/255) by construction,
    so E_k^2 = sum_{j>k} sigma_j^2 = q^k (1 - q^(256-k)) / (1 - q) with
    q = 10^(-8/255) (a geometric series).  The oracle's SVD of the dense
    matrix must recover the spectrum, and ||A - A_k||_F from its own factors
    must equal that closed form (Sec. 4, Eckart-Young)."""
    w = synth.matrix_small()
    A = w["A"]
    U, S, Vt = O.svd(A)
    sig = w["sigma"]
    np.testing.assert_allclose(S, sig, rtol=1e-12, atol=1e-15)
    q = 10.0 ** (-8.0 / 255.0)
    norm_a = math.sqrt((1 - q ** 256) / (1 - q))
    assert abs(np.linalg.norm(A) - norm_a) <= 1e-13 * norm_a
    for k in (20, 21):
        closed = math.sqrt(q ** k * (1 - q ** (256 - k)) / (1 - q))
        Ak = O.lowrank_dense(U[:, :k], S[:k], Vt[:k].T)
        assert abs(O.fro_diff(A, Ak) - closed) <= 1e-12 * closed
        assert abs(O.tail_norms(S)[k] - closed) <= 1e-12 * closed


def test_tail_norms_monotone_and_exact():
    sig = np.array([3.0, 2.0, 2.0, 1.0])
    E = O.tail_norms(sig)
    np.testing.assert_array_equal(E, [math.sqrt(18.0), 3.0, math.sqrt(5.0), 1.0, 0.0])
    s2 = synth.sigma_square(8192)
    E2 = O.tail_norms(s2)
    assert np.all(np.diff(E2) <= 0)


def test_tt_svd_recovers_exact_tt_rank():
    dims, ranks = (6, 7, 5, 4), (1, 3, 4, 2, 1)
    rng = np.random.default_rng([12969, 94, 0])
    cores = [rng.standard_normal((ranks[l], dims[l], ranks[l + 1])) for l in range(4)]
    T = O.tt_full(cores)
    rec = O.tt_svd(T, eps=1e-12)
    _, r = O.tt_shape(rec)
    assert r == list(ranks)
    assert O.fro_diff(O.tt_full(rec), T) <= 1e-13 * O.fro(T)
    # higher nominal ranks are capped by the valid unfolding dimensions
    big = O.tt_svd(T, ranks=[50, 50, 50])
    assert O.tt_shape(big)[1] == [1, 6, 20, 4, 1]
    assert O.fro_diff(O.tt_full(big), T) <= 1e-13 * O.fro(T)


def test_tt_svd_error_bound_and_capping():
    """||T - T_R|| <= (sum eps_l^2)^{1/2} (Sec. 5.1 eq. tt_svd_error), and the
    Salinas-A capping example of Sec. 7.4 (83 x 86 x 204, R_nom = 160 gives
    (83,160), R+ = 161 gives (83,161)) on a random tensor of that shape."""
    T = synth.decay_3d(30)
    for R in (2, 5, 9):
        cores = O.tt_svd(T, ranks=[R, R])
        # unfolding residuals of the best rank-R approximations
        eps2 = 0.0
        for l in (1, 2):
            M = T.reshape(int(np.prod(T.shape[:l])), -1)
            s = np.linalg.svd(M, compute_uv=False)
            eps2 += float(np.sum(s[R:] ** 2))
        assert O.fro_diff(O.tt_full(cores), T) <= math.sqrt(eps2) * (1 + 1e-12)
    rng = np.random.default_rng([12969, 94, 1])
    Ts = rng.standard_normal((83, 86, 204))
    assert O.tt_shape(O.tt_svd(Ts, ranks=[160, 160]))[1] == [1, 83, 160, 1]
    assert O.tt_shape(O.tt_svd(Ts, ranks=[161, 161]))[1] == [1, 83, 161, 1]


def test_left_orthogonalize_properties():
    rng = np.random.default_rng([12969, 94, 2])
    dims, ranks = (5, 6, 7, 4), (1, 4, 5, 3, 1)
    cores = [rng.standard_normal((ranks[l], dims[l], ranks[l + 1])) * (3.0 ** l) for l in range(4)]
    T = O.tt_full(cores)
    lo = O.left_orthogonalize(cores)
    assert O.fro_diff(O.tt_full(lo), T) <= 1e-13 * O.fro(T)
    for l in range(3):
        M = lo[l].reshape(-1, lo[l].shape[2])
        assert np.linalg.norm(M.T @ M - np.eye(M.shape[1])) <= 1e-13
    # TT-SVD output is already left-orthogonal: the gauge step changes
    # nothing beyond rounding (Sec. 7.2)
    cs = O.tt_svd(synth.decay_3d(20), ranks=[6, 6])
    lo2 = O.left_orthogonalize(cs)
    for a, b in zip(cs, lo2):
        assert np.max(np.abs(a - b)) <= 1e-13 * max(1.0, np.max(np.abs(a)))


def test_tt_svd_memo_is_bitwise_transparent():
    """The SVD memo only reuses the SVD of an unfolding that an earlier run
    on the same tensor already computed for the same kept ranks: cores are
    identical bit for bit to fresh runs, and the first unfolding's SVD is
    computed once for every rank choice."""
    rng = np.random.default_rng([12969, 77])
    T = rng.standard_normal((6, 7, 8, 5))
    memo = {}
    for ranks in ([3, 4, 2], [3, 5, 2], [2, 4, 2], [3, 4, 3]):
        fresh = O.tt_svd(T, ranks=ranks)
        memod = O.tt_svd(T, ranks=ranks, svd_memo=memo)
        assert len(fresh) == len(memod)
        for a, b in zip(fresh, memod):
            assert a.shape == b.shape and np.array_equal(a.view(np.uint64), b.view(np.uint64))
    assert sum(1 for key in memo if key == ()) == 1
    assert {key for key in memo if len(key) == 1} == {(2,), (3,)}

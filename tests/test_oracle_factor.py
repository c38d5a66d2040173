"""Pins of the oracle's randomized factorizations (the end-to-end
decomposition left to future work in Sec. sec:conclusion; randomized range
finder of Halko, Martinsson and Tropp; TT-SVD of Sec. 5.1 with eq.
tt_svd_error).  Each result is checked against something the oracle does
not compute itself: numpy's LAPACK SVD, closed-form truncated SVDs, exact
low-rank reconstructions, and the oracle's own deterministic TT-SVD (pinned
to the paper's tables elsewhere) when the test vectors span the exact
dominant subspaces."""
import math

import numpy as np
import pytest

import oracle as O
from paper_2607_12969_amd import synth


def _lowrank(m, n, rho, seed):
    rng = np.random.default_rng([12969, 70, seed])
    return rng.standard_normal((m, rho)) @ rng.standard_normal((rho, n))


def _rel(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


@pytest.mark.parametrize("m,n,rho,l,k", [(40, 30, 5, 8, 5), (30, 47, 3, 3, 3), (64, 64, 20, 26, 20)])
def test_exact_low_rank_is_reproduced(m, n, rho, l, k):
    """rank(A) <= k: the sketch spans range(A), so U S Vt = A, and S equals
    LAPACK's singular values."""
    A = _lowrank(m, n, rho, m + n)
    U, S, Vt = O.randomized_svd(A, synth.test_vectors(l, n, 1), k)
    assert _rel((U * S) @ Vt, A) <= 1e-13
    ref = np.linalg.svd(A, compute_uv=False)[:k]
    assert np.max(np.abs(S - ref)) <= 1e-13 * ref[0]


@pytest.mark.parametrize("power_iters", [0, 2])
def test_dominant_subspace_sketch_gives_truncated_svd(power_iters):
    """Test vectors spanning the top-l right singular vectors: the result is
    the truncated SVD P_k diag(sigma_k) Q_k^T of the closed-form matrix."""
    m, n, k, l = 50, 40, 6, 9
    sigma = 2.0 ** -np.arange(n, dtype=np.float64)
    P = synth.haar(np.random.default_rng(5), m, n)
    Q = synth.haar(np.random.default_rng(6), n, n)
    A = (P * sigma) @ Q.T
    mix = synth.haar(np.random.default_rng(7), l, l)
    Omega = mix @ Q[:, :l].T                      # l rows spanning the top-l right subspace
    U, S, Vt = O.randomized_svd(A, Omega, k, power_iters)
    np.testing.assert_allclose(S, sigma[:k], rtol=1e-13, atol=0)
    best = (P[:, :k] * sigma[:k]) @ Q[:, :k].T
    assert _rel((U * S) @ Vt, best) <= 1e-13
    # the singular vectors themselves, up to sign
    sg = np.sign(np.sum(U * P[:, :k], axis=0))
    assert np.max(np.abs(U * sg - P[:, :k])) <= 1e-12
    assert np.max(np.abs(Vt.T * sg - Q[:, :k])) <= 1e-12


def test_power_iteration_equals_premultiplied_sketch():
    """One subspace iteration spans range(A A^T A Omega^T): the same result
    as no iteration on the test vectors (A^T A Omega^T)^T."""
    sigma = np.linspace(1.0, 0.02, 30)
    A = synth.spectral_matrix(45, 35, sigma, tag=3)
    Om = synth.test_vectors(12, 35, 3)
    U1, S1, V1 = O.randomized_svd(A, Om, 8, power_iters=1)
    U0, S0, V0 = O.randomized_svd(A, (A.T @ (A @ Om.T)).T, 8, power_iters=0)
    assert _rel((U1 * S1) @ V1, (U0 * S0) @ V0) <= 1e-10
    np.testing.assert_allclose(S1, S0, rtol=1e-10)


@pytest.mark.parametrize("power_iters", [0, 1])
def test_error_against_eckart_young(power_iters):
    """||A - U S Vt||_F is never below the optimal tail (Eckart-Young) and,
    with ten oversampling vectors on a 2^-j spectrum, within 1 % of it;
    U and V have orthonormal columns."""
    n, k, l = 60, 10, 20
    sigma = 2.0 ** -np.arange(n, dtype=np.float64)
    A = synth.spectral_matrix(80, n, sigma, tag=4)
    U, S, Vt = O.randomized_svd(A, synth.test_vectors(l, n, 4), k, power_iters)
    err = np.linalg.norm(A - (U * S) @ Vt)
    opt = math.sqrt(float(np.sum(sigma[k:] ** 2)))
    assert opt * (1 - 1e-12) <= err <= 1.01 * opt
    assert np.linalg.norm(U.T @ U - np.eye(k)) <= 1e-13
    assert np.linalg.norm(Vt @ Vt.T - np.eye(k)) <= 1e-13


def test_argument_errors():
    A = np.ones((10, 8))
    with pytest.raises(ValueError):
        O.randomized_svd(A, np.ones((4, 7)), 2)      # wrong sketch length
    with pytest.raises(ValueError):
        O.randomized_svd(A, np.ones((4, 8)), 5)      # k > l
    with pytest.raises(ValueError):
        O.randomized_svd(A, np.ones((9, 8)), 2)      # l > min(m, n)


def _exact_tt(dims, ranks, seed):
    rng = np.random.default_rng([12969, 71, seed])
    cores = [rng.standard_normal((ranks[l], dims[l], ranks[l + 1])) for l in range(len(dims))]
    return O.tt_full(cores)


@pytest.mark.parametrize("dims,ranks", [((6, 5, 4), (2, 3)), ((4, 5, 3, 6), (3, 5, 4)), ((3, 4, 5, 2, 3), (2, 4, 3, 2))])
def test_tt_exact_ranks_are_reproduced(dims, ranks):
    """A tensor of exact TT ranks: reproduced, and step l's singular values
    are those of the unfolding T_(l) (prod_{i<=l} n_i x rest, LAPACK)."""
    T = _exact_tt(dims, (1,) + ranks + (1,), len(dims))
    oms = []
    r_prev = 1
    for l, r in enumerate(ranks):
        cols = int(np.prod(dims[l + 1:]))
        oms.append(synth.test_vectors(min(r + 2, cols, r_prev * dims[l]), cols, 10 + l))
        r_prev = r
    cores, info = O.tt_svd_randomized(T, ranks, oms)
    assert O.tt_shape(cores)[1] == [1, *ranks, 1]
    assert _rel(O.tt_full(cores), T) <= 1e-12
    for l, r in enumerate(ranks):
        ref = np.linalg.svd(T.reshape(int(np.prod(dims[:l + 1])), -1), compute_uv=False)[:r]
        np.testing.assert_allclose(info["sigma"][l], ref, rtol=1e-11)
    # left-orthonormal unfoldings
    for c in cores[:-1]:
        M = c.reshape(-1, c.shape[2])
        assert np.linalg.norm(M.T @ M - np.eye(M.shape[1])) <= 1e-13


def test_tt_dominant_subspace_sketch_gives_tt_svd():
    """Test vectors spanning each unfolding's top right singular subspace
    (taken from the oracle's deterministic TT-SVD, itself pinned to the
    paper's tables): the randomized run is that TT-SVD."""
    T = synth.decay_3d(14)
    ranks = [5, 5]
    det = O.tt_svd(T, ranks=ranks)
    # the unfoldings the deterministic run factors, and their right singular vectors
    C1 = T.reshape(14, -1)
    _, _, Vt1 = np.linalg.svd(C1, full_matrices=False)
    C2 = (det[0].reshape(14, 5).T @ C1).reshape(5 * 14, 14)
    _, _, Vt2 = np.linalg.svd(C2, full_matrices=False)
    oms = [Vt1[:8], Vt2[:8]]
    cores, _ = O.tt_svd_randomized(T, ranks, oms)
    assert _rel(O.tt_full(cores), O.tt_full(det)) <= 1e-12


def test_tt_error_bound():
    """eq. tt_svd_error with the realized step errors: eps_1 <= ||T - T_R||
    <= (sum eps_l^2)^(1/2) (every step is an orthogonal projection)."""
    T = synth.decay_3d(16) + 1e-3 * np.random.default_rng(9).standard_normal((16, 16, 16))
    oms = [synth.test_vectors(9, 256, 20), synth.test_vectors(9, 16, 21)]
    cores, info = O.tt_svd_randomized(T, [6, 6], oms)
    E = O.fro_diff(T, O.tt_full(cores))
    eps = info["step_err"]
    assert eps[0] * (1 - 1e-12) <= E <= math.sqrt(sum(e * e for e in eps)) * (1 + 1e-12)

"""CPU checks of the parity checkers themselves (no GPU): the componentwise
bounds of Lemma lem:dot (Sec. 5.2) hold for honest low-precision
evaluations of the apply and the TT chain done here with numpy in FP32 /
FP16, and the checks reject results with a fault planted on the CPU (a sign
flip, one zeroed entry, two swapped rows) that the global Frobenius norm can
miss."""
import numpy as np
import pytest

import oracle as O
from paper_2607_12969_amd import synth
from parity import (NP_DTYPES, TOL, apply_bound, componentwise_ratio, rel_fro, stored_pair, tile_rel_fro_max,
                    tt_bound)


def _honest_apply(u, s, v, x, prec):
    """Two phases with FP32 sums (FP64 for fp64), T' rounded to the storage
    type, the output rounded to it: what the kernels are allowed to do."""
    acc = np.float64 if prec == "fp64" else np.float32
    T = (v.astype(acc).T @ x.astype(acc)) * s.astype(acc)[:, None]
    T = T.astype(NP_DTYPES[prec]).astype(acc)
    return (u.astype(acc) @ T).astype(NP_DTYPES[prec]).astype(np.float64)


@pytest.mark.parametrize("prec", ["fp64", "fp32", "fp16"])
def test_apply_checks_accept_honest_and_reject_planted(prec):
    d = synth.random_factors(640, 300, 41, 192, tag=31)
    hs = [stored_pair(a, prec) for a in (d["U"], d["s"], d["V"], d["X"])]
    u, s, v, x = [o for _, o in hs]
    ref = O.apply(u, s, v, x)
    bound = apply_bound(u, s, v, x, prec, ref)
    Y = _honest_apply(u, s, v, x, prec)
    assert componentwise_ratio(Y, ref, bound) <= 1.0
    assert rel_fro(Y, ref) <= TOL[prec] and tile_rel_fro_max(Y, ref) <= TOL[prec]
    i, j = np.unravel_index(np.argmax(np.abs(ref)), ref.shape)
    flip = Y.copy()
    flip[i, j] = -flip[i, j]
    assert componentwise_ratio(flip, ref, bound) > 1.0
    zero = Y.copy()
    zero[333, 77] = 0.0                      # one typical entry lost
    assert tile_rel_fro_max(zero, ref) > TOL[prec]
    swap = Y.copy()
    swap[[100, 101]] = swap[[101, 100]]      # a row-index fault
    assert componentwise_ratio(swap, ref, bound) > 1.0


def _honest_tt(cores, prec):
    """Left-to-right chain with FP32 sums (FP64 for fp64), every interface
    rounded once to the storage type, output rounded to it."""
    acc = np.float64 if prec == "fp64" else np.float32
    Z = cores[0].astype(acc).reshape(-1, cores[0].shape[2])
    for c in cores[1:]:
        Z = Z.astype(NP_DTYPES[prec]).astype(acc)
        r0, n, r1 = c.shape
        Z = (Z @ c.astype(acc).reshape(r0, n * r1)).reshape(-1, r1)
    dims = [int(c.shape[1]) for c in cores]
    return Z.astype(NP_DTYPES[prec]).astype(np.float64).reshape(dims)


@pytest.mark.parametrize("prec", ["fp64", "fp32", "fp16"])
@pytest.mark.parametrize("dims,ranks", [((30, 40, 50), (1, 12, 17, 1)), ((6, 7, 5, 9), (1, 5, 9, 6, 1))])
def test_tt_checks_accept_honest_and_reject_planted(prec, dims, ranks):
    cores = synth.random_tt_cores(dims, ranks, tag=sum(dims))
    st = [stored_pair(c, prec)[1] for c in cores]
    ref = O.tt_full(st)
    bound = tt_bound(st, prec, ref)
    got = _honest_tt(st, prec)
    assert componentwise_ratio(got, ref, bound) <= 1.0
    assert rel_fro(got, ref) <= TOL[prec]
    flip = got.copy().ravel()
    q = int(np.argmax(np.abs(ref)))
    flip[q] = -flip[q]
    assert componentwise_ratio(flip.reshape(ref.shape), ref, bound) > 1.0


def test_fp16_subnormal_outputs_fit_the_floor():
    """Outputs far below the binary16 normal range (the situation of an
    unnormalized 16^6 train) carry absolute errors up to half the
    subnormal spacing; the bound's floor admits exactly the rounding and
    nothing of the output's size."""
    cores = [c * 0.01 for c in synth.random_tt_cores((20, 30, 40), (1, 6, 7, 1), tag=3)]
    st = [stored_pair(c, "fp16")[1] for c in cores]
    ref = O.tt_full(st)
    assert np.mean(np.abs(ref) < 2.0 ** -14) > 0.5      # mostly subnormal in binary16
    bound = tt_bound(st, "fp16", ref)
    assert componentwise_ratio(_honest_tt(st, "fp16"), ref, bound) <= 1.0
    assert componentwise_ratio(np.zeros_like(ref), ref, bound) > 1.0

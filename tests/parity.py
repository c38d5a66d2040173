"""Helpers shared by the GPU parity tests: rounding of seeded FP64 inputs to
the storage precision (numpy's correctly rounded casts; the oracle's own
rounding is checked to give the same bits), transfers, and the relative
Frobenius error used by every tolerance."""
import math

import numpy as np

import oracle as O

NP_DTYPES = {"fp64": np.float64, "fp32": np.float32, "fp16": np.float16}
# relative Frobenius tolerances against the oracle on the same stored values
TOL = {"fp64": 1e-12, "fp32": 1e-5, "fp16": 2e-3}
PRECS = ("fp64", "fp32", "fp16")


def stored_pair(x, prec):
    """(array in the storage dtype for the GPU, its exact FP64 value for the
    oracle).  The GPU copy is rounded by numpy, the oracle copy by the
    oracle's own RNE routine; the two must agree bit for bit."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    h = x.astype(NP_DTYPES[prec])
    o = O.round_to(x, prec)
    if prec != "fp64":
        bits = {"fp32": np.uint32, "fp16": np.uint16}[prec]
        assert np.array_equal(h.view(bits), o.view(bits)), "roundings disagree"
    return h, O.widen(o)


def to_dev(a, device="cuda:0"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def rel_fro(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = math.sqrt(O.fro(ref) ** 2) if ref.size else 0.0
    num = O.fro_diff(got.ravel(), ref.ravel())
    return num / den if den > 0 else num


# ---- componentwise bounds (Lemma lem:dot, Sec. 5.2) -------------------------
# unit roundoff of the accumulation and of the storage format
U_ACC = {"fp64": 2.0 ** -53, "fp32": 2.0 ** -24, "fp16": 2.0 ** -24}
U_STO = {"fp64": 2.0 ** -53, "fp32": 2.0 ** -24, "fp16": 2.0 ** -11}
# largest absolute error of one rounding into the storage format near zero
# (half the spacing of its subnormals)
ABS_FLOOR = {"fp64": 2.0 ** -1075, "fp32": 2.0 ** -150, "fp16": 2.0 ** -25}


def gamma(count, u):
    """gamma_m = m u / (1 - m u) of Lemma lem:dot."""
    return count * u / (1.0 - count * u)


def apply_bound(u, s, v, x, prec, ref):
    """Componentwise bound on |Y_hat - Y| for the two-phase apply, from
    Lemma lem:dot applied to both phases on the stored values:
      phase 1: |T_hat - V^T X| <= gamma_n |V|^T |X|  (any summation order);
      scaling: one rounding in the accumulation format, plus for FP16 the
               rounding of T' to binary16 (relative u_s, absolute floor);
      phase 2: |fl(U T') - U T'| <= gamma_k |U| |T'|;
      output:  one rounding to the storage format (u_s |Y| + floor).
    Summed to first order with G = |U| |diag(s)| |V|^T |X| (the oracle's FP64
    apply of the absolute values); matrix-core sums are allowed twice the
    unit roundoff per operation, and the oracle's own FP64 sums are added."""
    n, k = v.shape
    ua, us = U_ACC[prec], U_STO[prec]
    t_round = ua + (us if prec == "fp16" else 0.0)
    c = 1.01 * (gamma(n, 2 * ua) + gamma(k, 2 * ua) + t_round) * (1.0 + us) + gamma(n + k, 2.0 ** -53)
    G = O.apply(np.abs(u), np.abs(s), np.abs(v), np.abs(x))
    floor_t = ABS_FLOOR[prec] if prec == "fp16" else 0.0
    rows_u = np.abs(u).sum(axis=1, keepdims=True)          # |U| 1: spread of T' floors into Y
    return us * np.abs(ref) + c * G + ABS_FLOOR[prec] + 1.01 * floor_t * rows_u


def tt_bound(cores, prec, ref):
    """Componentwise bound on |T_hat - T| for the left-to-right chain
    (Sec. 5.2: gamma |G_1(i_1)| ... |G_d(i_d)|, by Lemma lem:dot at every
    contraction): each level's K-term sums (gamma_{r_{l-1}}), every interface
    possibly rounded once to the storage format (relative u_s plus a floor
    carried through the remaining cores), and the output rounding."""
    d = len(cores)
    ua, us = U_ACC[prec], U_STO[prec]
    acc = sum(gamma(int(c.shape[0]), 2 * ua) for c in cores[1:])
    inter = (d - 1) * (ua + (us if prec == "fp16" else 0.0))
    c = 1.01 * (acc + inter) * (1.0 + us) + gamma(sum(int(cc.shape[0]) for cc in cores), 2.0 ** -53)
    absc = [np.abs(cc) for cc in cores]
    bound = us * np.abs(ref) + c * O.tt_full(absc) + ABS_FLOOR[prec]
    if prec == "fp16":
        dims = [int(cc.shape[1]) for cc in cores]
        for l in range(1, d):
            # a floor on interface Z_l (rank r_l) reaches the output through |G_{l+1}| ... |G_d|
            ones = np.ones((1, 1, int(cores[l].shape[0])))
            tail = O.tt_full([ones] + absc[l:]).reshape([1] * l + dims[l:])
            bound = bound + 1.01 * ABS_FLOOR[prec] * tail
    return bound


def componentwise_ratio(got, ref, bound):
    """max |got - ref| / bound over all entries (<= 1 passes)."""
    got = np.asarray(got, dtype=np.float64)
    return float(np.max(np.abs(got - ref) / bound)) if got.size else 0.0


def tile_rel_fro_max(got, ref, tile=64):
    """Largest relative Frobenius error over the tile x tile blocks of a
    matrix (ragged edge blocks included): a fault confined to a few tiles of
    a large output cannot hide in the global norm."""
    got = np.asarray(got, dtype=np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, dtype=np.float64).reshape(got.shape)
    m, n = ref.shape
    tm, tn = -(-m // tile), -(-n // tile)
    pad = ((0, tm * tile - m), (0, tn * tile - n))
    d2 = np.pad((got - ref) ** 2, pad).reshape(tm, tile, tn, tile).sum(axis=(1, 3))
    r2 = np.pad(ref ** 2, pad).reshape(tm, tile, tn, tile).sum(axis=(1, 3))
    ok = r2 > 0
    worst = np.sqrt(d2[ok] / r2[ok]).max() if ok.any() else 0.0
    return float(max(worst, np.sqrt(d2[~ok]).max() if (~ok).any() else 0.0))

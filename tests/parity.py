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

"""The allocation-free apply (lrc_matrix_apply_noalloc) against the ordinary
entry point: the same kernels and plan over a scratch array the library
holds per device, so the outputs must be identical bit for bit, and both
within the parity tolerances of the oracle.  Two calls in a row, the second
smaller, for every precision and both kernel pairs (the second call runs
over what the first left in the scratch)."""
import numpy as np
import pytest

import oracle as O
from paper_2607_12969_amd import synth
from parity import TOL, rel_fro, stored_pair, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def lrc():
    import torch
    from paper_2607_12969_amd import lrc as mod
    assert torch.cuda.is_available()
    mod.lib()
    yield mod
    mod.set_apply_path(mod.PATH_AUTO)


def _both(lrc, shape, prec, path, tag):
    import torch
    m, n, k, b = shape
    d = synth.random_factors(m, n, k, b, tag=tag)
    hs = [stored_pair(a, prec) for a in (d["U"], d["s"], d["V"], d["X"])]
    dv = [to_dev(h) for h, _ in hs]
    lrc.set_apply_path(path)
    try:
        ref_gpu = lrc.matrix_apply(*dv)
        Y = torch.full((m, b), float("nan"), dtype=dv[0].dtype, device=dv[0].device)
        lrc.matrix_apply_noalloc(*dv, Y)
        torch.cuda.synchronize()
    finally:
        lrc.set_apply_path(lrc.PATH_AUTO)
    got, want = Y.cpu().numpy(), ref_gpu.cpu().numpy()
    assert np.array_equal(got.view(np.uint8), want.view(np.uint8)), (shape, prec, path)
    u, s, v, x = [o for _, o in hs]
    assert rel_fro(got.astype(np.float64), O.apply(u, s, v, x)) <= TOL[prec]


@pytest.mark.parametrize("prec", ["fp64", "fp32", "fp16"])
@pytest.mark.parametrize("path", [1, 2])
def test_noalloc_matches_apply_two_calls(lrc, prec, path):
    big = (3000, 2000, 65, 8 if path == 1 else 300)
    small = (700, 500, 21, 3 if path == 1 else 70)
    print(f"noalloc prec={prec} path={path} {big} then {small}", flush=True)
    _both(lrc, big, prec, path, tag=41)
    _both(lrc, small, prec, path, tag=42)


def test_noalloc_rejects_oversize_before_launch(lrc):
    """65536 x 4096 at rank 512 and batch 20000: T' alone is 82 MB, above the
    scratch; the call fails on the host before anything is launched (the
    addresses are disjoint placeholders that are never dereferenced)."""
    import torch
    ptrs = [0x10000, 0x20000, 0x30000, 0x40000, 0x90000000]
    with pytest.raises(lrc.LrcError, match="scratch"):
        lrc._check(lrc.lib().lrc_matrix_apply_noalloc(*ptrs, 65536, 4096, 512, 20000, lrc.FP64))
    torch.cuda.synchronize()

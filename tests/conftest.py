import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
    config.addinivalue_line("markers", "slow: takes more than a few seconds on the CPU")


def read_golden(name):
    """Rows of a CSV fixture under tests/golden/ ('#' lines are comments)."""
    import csv
    path = os.path.join(ROOT, "tests", "golden", name)
    with open(path) as fh:
        lines = [ln for ln in fh if not ln.startswith("#")]
    return list(csv.DictReader(lines))


@pytest.fixture(scope="session")
def hyper():
    """The normalized 512 x 512 x 224 hyperspectral-shaped cube and its own
    fixed-rank TT-SVD (the oracle's, one SVD memo for every schedule): FP64
    bases at (64, 64) and (32, 32); compensated trains at (65, 65), (33, 33)
    and (36, 36), left-orthogonalized.  Shared by the reconstruction and
    certificate tests (the oracle's SVD of the 512 x 114688 unfolding takes
    tens of seconds)."""
    import oracle as O
    from paper_2607_12969_amd import synth
    T = synth.hyperspectral()
    memo = {}
    base = {r: O.tt_svd(T, ranks=[r, r], svd_memo=memo) for r in (64, 32)}
    aug = {r: O.left_orthogonalize(O.tt_svd(T, ranks=[r, r], svd_memo=memo)) for r in (65, 33, 36)}
    return T, base, aug

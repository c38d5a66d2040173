"""Apply parity with the matrix-core tile edge pinned by LRC_APPLY_TILE (64
or 128), on shapes whose tiles are mostly edges.  The library reads the
variable once per process, so test_gpu_apply.py runs this file in a child
process with the variable set; exit status 0 when every case is within the
tolerances of the parity tests (relative Frobenius error and the
componentwise bound of Lemma lem:dot, Sec. 5.2)."""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
for p in (HERE, os.path.dirname(HERE)):
    if p not in sys.path:
        sys.path.insert(0, p)

import numpy as np  # noqa: E402

import oracle as O  # noqa: E402
from paper_2607_12969_amd import lrc, synth  # noqa: E402
from parity import PRECS, TOL, apply_bound, componentwise_ratio, rel_fro, stored_pair, to_dev  # noqa: E402

CASES = [(300, 200, 129, 70), (1000, 700, 65, 129), (129, 4100, 100, 200), (700, 900, 257, 300),
         (200, 300, 37, 130), (1100, 520, 513, 260)]


def main():
    import torch
    assert torch.cuda.is_available()
    lrc.lib()
    lrc.set_apply_path(lrc.PATH_MFMA)
    bad = 0
    for m, n, k, b in CASES:
        d = synth.random_factors(m, n, k, b, tag=m * 5 + n * 3 + k + b)
        for prec in PRECS:
            hs = [stored_pair(a, prec) for a in (d["U"], d["s"], d["V"], d["X"])]
            Y = lrc.matrix_apply(*[to_dev(h) for h, _ in hs])
            torch.cuda.synchronize()
            Y = Y.cpu().numpy().astype(np.float64)
            u, s, v, x = [o for _, o in hs]
            ref = O.apply(u, s, v, x)
            err = rel_fro(Y, ref)
            cw = componentwise_ratio(Y, ref, apply_bound(u, s, v, x, prec, ref))
            ok = err <= TOL[prec] and cw <= 1.0
            bad += not ok
            print(f"tile={os.environ.get('LRC_APPLY_TILE')} m={m} n={n} k={k} b={b} {prec}: "
                  f"rel {err:.3e} componentwise {cw:.3f} {'ok' if ok else 'FAIL'}", flush=True)
    lrc.set_apply_path(lrc.PATH_AUTO)
    return 1 if bad else 0


if __name__ == "__main__":
    sys.exit(main())

"""The matrix-core ceiling probe (a measurement aid for the roofline
fractions): each precision's register-only MFMA loop must land between a
third of the published MI355X peak and slightly above it (clocks vary)."""
import pytest

pytestmark = pytest.mark.gpu

PEAK = {"fp64": 78.6, "fp32": 157.3, "fp16": 2500.0}


@pytest.mark.parametrize("prec", ["fp64", "fp32", "fp16"])
def test_mfma_ceiling_near_published_peak(prec):
    import torch
    from paper_2607_12969_amd import lrc
    assert torch.cuda.is_available()
    t = lrc.mfma_ceiling(prec)
    print(f"mfma ceiling {prec}: {t:.1f} TFLOP/s", flush=True)
    assert PEAK[prec] / 3 < t < 1.1 * PEAK[prec]

"""Host-side checks of the Python binding (no GPU needed): shapes, dtypes and
caller-supplied outputs are validated before any tensor reaches the device
check or the C ABI, so a wrong-size output buffer can never be handed to a
kernel."""
import pytest

torch = pytest.importorskip("torch")

from paper_2607_12969_amd import lrc  # noqa: E402


def _apply_args(m=12, n=10, k=3, b=4, dtype=torch.float32):
    return [torch.zeros(m, k, dtype=dtype), torch.zeros(k, dtype=dtype), torch.zeros(n, k, dtype=dtype),
            torch.zeros(n, b, dtype=dtype)]


def test_apply_rejects_wrong_output_buffer():
    U, s, V, X = _apply_args()
    with pytest.raises(ValueError, match="Y has shape"):
        lrc.matrix_apply(U, s, V, X, Y=torch.zeros(12, 5))          # batch 4, not 5
    with pytest.raises(ValueError, match="Y has shape"):
        lrc.matrix_apply(U, s, V, X, Y=torch.zeros(11, 4))
    with pytest.raises(ValueError, match="Y has dtype"):
        lrc.matrix_apply(U, s, V, X, Y=torch.zeros(12, 4, dtype=torch.float16))


def test_apply_rejects_inconsistent_factors():
    U, s, V, X = _apply_args()
    with pytest.raises(ValueError, match="shape mismatch"):
        lrc.matrix_apply(U, s, torch.zeros(9, 3), X)
    with pytest.raises(ValueError, match="shape mismatch"):
        lrc.matrix_apply(U, torch.zeros(4), V, X)
    with pytest.raises(TypeError):
        lrc.matrix_apply(U, s.double(), V, X)
    with pytest.raises(ValueError, match="on the GPU"):
        lrc.matrix_apply(U, s, V, X)                                 # consistent, but host tensors


def test_tt_rejects_wrong_output_and_train():
    cores = [torch.zeros(1, 4, 3), torch.zeros(3, 5, 2), torch.zeros(2, 6, 1)]
    with pytest.raises(ValueError, match="entries"):
        lrc.tt_reconstruct(cores, out=torch.zeros(4, 5, 5))
    with pytest.raises(ValueError, match="dtype"):
        lrc.tt_reconstruct(cores, out=torch.zeros(4, 5, 6, dtype=torch.float64))
    bad = [torch.zeros(1, 4, 3), torch.zeros(2, 5, 2), torch.zeros(2, 6, 1)]
    with pytest.raises(ValueError, match="rank"):
        lrc.tt_reconstruct(bad)
    with pytest.raises(ValueError, match="boundary"):
        lrc.tt_reconstruct([torch.zeros(2, 4, 3), torch.zeros(3, 5, 1)])


def _cert_factors(m=12, n=10, k=3, prec=torch.float16):
    f64 = [torch.zeros(m, k + 1, dtype=torch.float64), torch.zeros(k + 1, dtype=torch.float64),
           torch.zeros(n, k + 1, dtype=torch.float64)]
    return f64, [t.to(prec) for t in f64]


def test_certify_matrix_checks_factor_shapes():
    f64, low = _cert_factors()
    sig = [1.0 - 0.05 * j for j in range(10)]
    with pytest.raises(ValueError, match="k \\+ 1"):
        lrc.certify_matrix(sig, *f64, *low, 4)                       # factors hold k + 1 = 4 columns, not 5
    with pytest.raises(ValueError, match="min\\(m, n\\)"):
        lrc.certify_matrix(sig[:4], *f64, *low, 3)                   # truncated spectrum
    with pytest.raises(ValueError, match="Vh has shape"):
        lrc.certify_matrix(sig, *f64, low[0], low[1], low[2][:, :3], 3)
    with pytest.raises(TypeError, match="float64"):
        lrc.certify_matrix(sig, f64[0].float(), f64[1], f64[2], *low, 3)
    with pytest.raises(ValueError, match="A has shape"):
        lrc.certify_matrix(sig, *f64, *low, 3, A=torch.zeros(10, 12, dtype=torch.float64))


def test_certify_tt_checks_trains():
    dims = (4, 5, 6)
    base = [torch.zeros(1, 4, 2, dtype=torch.float64), torch.zeros(2, 5, 2, dtype=torch.float64),
            torch.zeros(2, 6, 1, dtype=torch.float64)]
    aug = [torch.zeros(1, 4, 3, dtype=torch.float64), torch.zeros(3, 5, 3, dtype=torch.float64),
           torch.zeros(3, 6, 1, dtype=torch.float64)]
    aug_h = [c.half() for c in aug]
    T = torch.zeros(dims, dtype=torch.float64)
    with pytest.raises(ValueError, match="T has"):
        lrc.certify_tt(torch.zeros(4, 5, 5, dtype=torch.float64), base, aug, aug_h)
    with pytest.raises(ValueError, match="stored core"):
        lrc.certify_tt(T, base, aug, [c.half() for c in base])
    with pytest.raises(ValueError, match="dims"):
        lrc.certify_tt(T, base, [aug[0], torch.zeros(3, 7, 3, dtype=torch.float64), aug[2]], aug_h)
    with pytest.raises(TypeError, match="float64"):
        lrc.certify_tt(T, [c.float() for c in base], aug, aug_h)
    with pytest.raises(ValueError, match="on the GPU"):
        lrc.certify_tt(T, base, aug, aug_h)                          # consistent, but host tensors


def test_mfma_ceiling_rejects_unknown_precision():
    with pytest.raises(ValueError, match="prec"):
        lrc.mfma_ceiling("bf16")

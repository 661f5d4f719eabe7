"""GPU results against properties the paper and linear algebra fix, without the
oracle's iteration: the limit of a convergent iteration (an SVD), the band the
constant triple maps singular values into, the sign of <X, O> and the trace
identity behind the Frobenius and Schatten-4 scales."""
import numpy as np
import pytest

from oracle import turbomuon as O
from gpu_helpers import from_device, log, make_input, relF, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402

TRIPLE = O.CONSTANT_TRIPLE
QUINTIC = (15 / 8, -10 / 8, 3 / 8)   # p(1) = 1, p'(1) = p''(1) = 0: converges to 1


def gpu_orth(X, dtype, iters, precond, coeffs=None):
    t = to_device(X, dtype)
    tm.orthogonalize(t, iters, coeffs, precond)
    torch.cuda.synchronize()
    return from_device(t)


def phi(x, coeffs):
    """p_t o ... o p_1 on scalars, p(x) = a x + b x^3 + c x^5."""
    for a, b, c in coeffs:
        x = a * x + b * x ** 3 + c * x ** 5
    return x


@pytest.mark.parametrize("dtype,tol", [("f32", 1e-4), ("bf16", 2e-2)])
@pytest.mark.parametrize("m,n", [(192, 640), (640, 192), (256, 256)])
def test_p2_limit_is_the_polar_factor_of_the_aol_input(dtype, tol, m, n):
    """Twenty steps of the convergent quintic from AOL(X) reach PolarFactor(AOL(X))
    (LAPACK SVD), which differs from PolarFactor(X) by the AOL bias (bias appendix)."""
    log(f"case: P2 {m}x{n} {dtype} AOL t=20 convergent quintic")
    X = make_input(m, n, 0.3, 11 + m, dtype)
    t = 20
    G = gpu_orth(X, dtype, t, "aol", [QUINTIC] * t)
    Qa = O.polar_factor(O.preconditioned(X, "aol"))
    e = relF(G, Qa)
    log(f"relF vs PolarFactor(AOL(X)) = {e:.3e}, bias = {O.eps_bias(X):.3e}")
    assert e <= tol
    if dtype == "f32":
        assert relF(G, O.polar_factor(X)) > 100 * e   # the limit is not PolarFactor(X)


@pytest.mark.parametrize("dtype,slack", [("f32", 1e-4), ("bf16", 5e-3)])
@pytest.mark.parametrize("m,n,precond", [(256, 1024, "aol"), (1024, 256, "aol"),
                                         (300, 300, "frobenius")])
def test_p4_output_singular_values_in_the_band(dtype, slack, m, n, precond):
    """An odd polynomial iteration maps each singular value sigma of X1 to phi(sigma):
    the output's singular values lie in phi([sigma_min(X1), sigma_max(X1)]) (dense 1-D
    sampling), up to the storage rounding.  Also <X, O> > 0 (Lemma 1)."""
    log(f"case: P4 {m}x{n} {dtype} {precond} t=4")
    X = make_input(m, n, 1.0, 5 + n, dtype)
    G = gpu_orth(X, dtype, 4, precond)
    sv1 = np.linalg.svd(O.preconditioned(X, precond), compute_uv=False)
    img = phi(np.linspace(sv1.min(), sv1.max(), 400001), [TRIPLE] * 4)
    lo, hi = img.min(), img.max()
    svg = np.linalg.svd(G, compute_uv=False)
    log(f"band [{lo:.4f}, {hi:.4f}], GPU sigma in [{svg.min():.4f}, {svg.max():.4f}]")
    assert svg.min() >= lo - slack and svg.max() <= hi + slack
    assert float(np.sum(X * G)) > 0


@pytest.mark.parametrize("dtype,tol", [("f32", 2e-6), ("bf16", 4e-3)])
@pytest.mark.parametrize("m,n", [(96, 300), (300, 96)])
def test_p8_trace_identity_ties_the_two_scales(dtype, tol, m, n):
    """The Frobenius scale comes from sums of squares of X, the Schatten-4 scale from
    sums of squares of the Gram A0.  With iters = 0 the outputs are X / ||X||_F and
    X / ||A0||_F^(1/2), and ||X||_F^2 = tr(A0): so ||X1_F||_F = 1 and
    ||X1_S4||_F^2 ||A0||_F = tr(A0).  For a rank-one X, ||A0||_F = tr(A0) and the
    two outputs coincide."""
    log(f"case: P8 {m}x{n} {dtype}")
    X = make_input(m, n, 0.8, 17, dtype)
    Y = X if m <= n else X.T
    A0 = Y @ Y.T
    F = gpu_orth(X, dtype, 0, "frobenius")
    S = gpu_orth(X, dtype, 0, "schatten4")
    assert abs(np.linalg.norm(F) - 1.0) <= tol
    lhs = np.linalg.norm(S) ** 2 * np.linalg.norm(A0)
    assert abs(lhs / np.trace(A0) - 1.0) <= 2 * tol
    rng = np.random.default_rng(3)
    from paper_2512_04632_amd import synth
    R1 = synth.cast(np.outer(rng.standard_normal(m), rng.standard_normal(n)), dtype)
    F1 = gpu_orth(R1, dtype, 0, "frobenius")
    S1 = gpu_orth(R1, dtype, 0, "schatten4")
    assert relF(S1, F1) <= tol

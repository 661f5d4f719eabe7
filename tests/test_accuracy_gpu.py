"""Polar error of the GPU path against the number of iterations (the trend of the
paper's polar-error figures, with the constant coefficient triple).

The GPU's bf16 result must track the fp64 oracle's polar error at every
iteration count, and the initialisation ordering of the pre-conditioning appendix
(AOL below Schatten-4 below Frobenius) must hold for the GPU results while the
iteration has not yet reached the triple's oscillation band (t <= 2)."""
import numpy as np
import pytest

from oracle import turbomuon as O
from paper_2512_04632_amd import synth
from gpu_helpers import BF16_TOL, log

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402


@pytest.mark.parametrize("n", [512, 1024])
def test_polar_error_sweep(n):
    """Prints one line per (pre-conditioning, t): the table of polar errors against
    iterations (run with -s to see it)."""
    X = synth.cast(synth.gaussian_matrix(n, n, seed=0), "bf16")
    Q = O.polar_factor(X)
    eps = {}
    for pre in ("frobenius", "schatten4", "aol"):
        for t in range(1, 7):
            g = torch.from_numpy(X.astype(np.float32)).to(torch.bfloat16).cuda()
            tm.orthogonalize(g, t, None, pre)
            torch.cuda.synchronize()
            G = g.float().cpu().numpy().astype(np.float64)
            R = O.orthogonalize(X, t, None, pre)
            eg, eo = O.eps_polar(G, X, Q), O.eps_polar(R, X, Q)
            log(f"{n}x{n} N(0,1) {pre:10s} t={t}: eps_polar gpu {eg:.4f} oracle {eo:.4f} "
                f"relF {O.rel_frobenius(G, R):.2e}")
            assert O.rel_frobenius(G, R) <= BF16_TOL
            assert abs(eg - eo) <= 0.05 * eo + 2e-3
            eps[pre, t] = eg
    for t in (1, 2):
        assert eps["aol", t] < eps["schatten4", t] < eps["frobenius", t]
    for pre in ("frobenius", "schatten4", "aol"):
        assert eps[pre, 2] < eps[pre, 1]

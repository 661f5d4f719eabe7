"""Shared helpers of the GPU tests: seeded inputs on the device and metrics."""
import sys

import numpy as np

from oracle import turbomuon as O
from paper_2512_04632_amd import synth

BF16_TOL = 2e-2        # relative Frobenius error of the bf16 path against the fp64 oracle
F32_TOL = 1e-4         # same for the fp32 path
EO_RATIO_TOL = 0.10    # bf16 polar error ||I - O O^T||_F / sqrt(k) within 10% of the oracle's


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def torch_dtype(name):
    import torch
    return torch.bfloat16 if name == "bf16" else torch.float32


def to_device(Xc, dtype):
    """float64 array of values exactly representable in dtype -> device tensor."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(Xc, dtype=np.float32)).to(torch_dtype(dtype)).cuda()


def from_device(t):
    return t.float().cpu().numpy().astype(np.float64)


def make_input(m, n, alpha, seed, dtype):
    return synth.cast(synth.power_law_matrix(m, n, alpha, seed), dtype)


def relF(G, R):
    return O.rel_frobenius(G, R)


def eo_ratio(G, R):
    return O.eps_ortho(G) / O.eps_ortho(R)


def block_relF_max(G, R, b=256):
    """Largest relative Frobenius error over the b x b blocks of the output (ragged
    edge blocks included), so that one wrong tile cannot hide in the global norm."""
    m, n = R.shape
    worst = 0.0
    for i in range(0, m, b):
        for j in range(0, n, b):
            worst = max(worst, O.rel_frobenius(G[i:i + b, j:j + b], R[i:i + b, j:j + b]))
    return worst


def normalised_quintic(a):
    """(a, b, c) with p(1) = 1 and p'(1) = 0 for p(x) = a x + b x^3 + c x^5:
    b = 5/2 - 2a, c = a - 3/2 (a = 15/8 is the convergent quintic)."""
    return (a, 2.5 - 2.0 * a, a - 1.5)


# A five-row coefficient schedule (decreasing a: the early rows grow small
# singular values fastest), built from the family above.
SCHEDULE5 = [normalised_quintic(a) for a in (3.0, 2.6, 2.2, 1.875, 1.6)]

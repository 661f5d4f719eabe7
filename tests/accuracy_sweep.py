"""Polar error against the number of iterations: the GPU's bf16 result and the
fp64 oracle on the same rounded N x N N(0,1) matrix, for the Frobenius,
Schatten-4 and AOL pre-conditionings and t = 1..6 with the constant triple.

Run on a GPU:  python tests/accuracy_sweep.py 1024   (one JSON line)
tests/test_accuracy_gpu.py checks the same sweep at N = 512.
"""
import json
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

from oracle import turbomuon as O  # noqa: E402
from paper_2512_04632_amd import synth  # noqa: E402


def sweep(n):
    import torch
    from paper_2512_04632_amd import _lib as tm
    X = synth.cast(synth.gaussian_matrix(n, n, seed=0), "bf16")
    Q = O.polar_factor(X)
    rows = []
    for pre in ("frobenius", "schatten4", "aol"):
        for t in range(1, 7):
            g = torch.from_numpy(X.astype(np.float32)).to(torch.bfloat16).cuda()
            tm.orthogonalize(g, t, None, pre)
            torch.cuda.synchronize()
            G = g.float().cpu().numpy().astype(np.float64)
            R = O.orthogonalize(X, t, None, pre)
            rows.append({"precond": pre, "iters": t, "eps_polar_gpu": round(O.eps_polar(G, X, Q), 4),
                         "eps_polar_oracle": round(O.eps_polar(R, X, Q), 4),
                         "rel_frobenius": round(O.rel_frobenius(G, R), 5)})
    return {"metric": "polar error vs iterations", "matrix": f"{n}x{n} N(0,1) bf16, seed 0",
            "coefficients": "constant (3.4445, -4.7750, 2.0315)", "rows": rows}


if __name__ == "__main__":
    print(json.dumps(sweep(int(sys.argv[1]) if len(sys.argv) > 1 else 1024)), flush=True)

"""Seeded synthetic gradient-like matrices.

This module only draws inputs; it contains none of the orthogonalization
arithmetic, so both the fp64 oracle and the HIP path can consume its output.

Recipe (one matrix of shape m x n, k = min(m, n), spectrum exponent alpha):

    X = U diag(sigma) V^T + 0.01 * E,     sigma_j = j^(-alpha), j = 1..k

* U (m x k) and V (n x k) have orthonormal columns drawn from the Haar
  measure: QR of a standard Gaussian matrix with the sign of R's diagonal
  folded into Q.
* E is i.i.d. N(0, 1).
* Everything is drawn in float64 from ``numpy.random.default_rng(seed)`` in
  the fixed order G_U, G_V, E, then cast once (round to nearest even) to the
  storage dtype.  Consumers compare against the *cast* values.

The paper draws its synthetic matrices from N(0, 1) (Sections 3.1 and 3.2)
and from heavy-tailed Levy laws (the appendix on realistic gradients); the
power-law-plus-noise matrices here stand in for real gradient matrices.
"""
from __future__ import annotations

import numpy as np

_BF16_DTYPES = ("bf16", "bfloat16")


def _haar_columns(rng: np.random.Generator, rows: int, cols: int) -> np.ndarray:
    g = rng.standard_normal((rows, cols))
    q, r = np.linalg.qr(g, mode="reduced")
    d = np.sign(np.diag(r))
    d[d == 0] = 1.0
    return q * d[None, :]


def power_law_matrix(m: int, n: int, alpha: float, seed: int,
                     noise: float = 0.01) -> np.ndarray:
    """float64 m x n matrix U diag(j^-alpha) V^T + noise * N(0,1)."""
    rng = np.random.default_rng(seed)
    k = min(m, n)
    u = _haar_columns(rng, m, k)
    v = _haar_columns(rng, n, k)
    sigma = np.arange(1, k + 1, dtype=np.float64) ** (-float(alpha))
    e = rng.standard_normal((m, n))
    return (u * sigma[None, :]) @ v.T + noise * e


def gaussian_matrix(m: int, n: int, seed: int) -> np.ndarray:
    """float64 m x n matrix with i.i.d. N(0, 1) entries."""
    return np.random.default_rng(seed).standard_normal((m, n))


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (nearest even), returned as float64.

    The value is first rounded to float32 (nearest even), then to bfloat16 by
    integer round-half-to-even on the float32 bit pattern.  Double rounding
    through float32 can differ from a direct float64 -> bf16 rounding only in
    ties of the float32 intermediate; the storage value is what both sides
    consume, so the exact rule only has to be applied consistently.
    """
    f = np.ascontiguousarray(x, dtype=np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    nan = np.isnan(f)
    out = rounded.astype(np.uint32).view(np.float32).astype(np.float64)
    out[nan] = np.nan
    return out


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """uint16 bit patterns of values that are already exactly bf16."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)


def cast(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round once to the storage dtype; returns float64 holding the stored values."""
    if dtype in _BF16_DTYPES:
        return round_to_bf16(x)
    if dtype in ("f32", "fp32", "float32"):
        return x.astype(np.float32).astype(np.float64)
    if dtype in ("f64", "fp64", "float64"):
        return np.array(x, dtype=np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


def block_diagonal_layout(m: int, n: int, count: int):
    """Split an m x n matrix into `count` blocks along its diagonal.

    Rows and columns are each cut into `count` runs whose lengths differ by at
    most one (the longer runs first); block i covers rows [r0, r1) and columns
    [c0, c1) of run i.  Returns a list of (r0, r1, c0, c1).  Every block has
    the orientation of the whole matrix (no taller than wide when m <= n, taller
    than wide otherwise), so a per-block computation that picks its side from
    the shape picks the same side as the whole.
    """
    if not (1 <= count <= min(m, n)):
        raise ValueError("count must be in 1..min(m, n)")

    def runs(total):
        q, r = divmod(total, count)
        edges = [0]
        for i in range(count):
            edges.append(edges[-1] + q + (1 if i < r else 0))
        return edges

    re, ce = runs(m), runs(n)
    out = [(re[i], re[i + 1], ce[i], ce[i + 1]) for i in range(count)]
    for r0, r1, c0, c1 in out:
        if (m <= n) != (r1 - r0 <= c1 - c0):
            raise ValueError(f"block {r1 - r0} x {c1 - c0} is not oriented as {m} x {n}")
    return out


def block_diagonal_blocks(m: int, n: int, count: int, alpha: float, seed: int):
    """Layout and float64 contents of a block-diagonal m x n input.

    Block i is ``power_law_matrix`` of its shape with seed ``seed + i``; every
    entry outside the blocks is zero.
    """
    layout = block_diagonal_layout(m, n, count)
    blocks = [power_law_matrix(r1 - r0, c1 - c0, alpha, seed + i)
              for i, (r0, r1, c0, c1) in enumerate(layout)]
    return layout, blocks


# Workloads: (count, m, n, alpha).  Matrix i of a workload, counted across
# its entries in the listed order, uses seed = base + i.
WORKLOADS = {
    # one 256 x 256 fp32 matrix, power law exponent 1.0
    "single_256_f32": {"dtype": "f32", "entries": [(1, 256, 256, 1.0)]},
    # one GPT-2-small MLP-shaped 768 x 3072 bf16 matrix, exponent 0.8
    "gpt2_mlp_768x3072": {"dtype": "bf16", "entries": [(1, 768, 3072, 0.8)]},
    # the 72 weight-shaped gradients of a 12-layer 768-wide transformer:
    # per layer 4 attention 768 x 768, one 768 x 3072 and one 3072 x 768
    "gpt2_small_12layer": {"dtype": "bf16", "entries":
                           [(48, 768, 768, 0.8), (12, 768, 3072, 0.8),
                            (12, 3072, 768, 0.8)]},
    # 8B-class transformer layer shapes, exponent 0.5
    "llm8b_4096x4096_b8": {"dtype": "bf16", "entries": [(8, 4096, 4096, 0.5)]},
    "llm8b_4096x14336_b8": {"dtype": "bf16", "entries": [(8, 4096, 14336, 0.5)]},
    # ResNet-style 3x3 conv gradients reshaped to out x (in * 9), exponent 1.0
    "resnet_conv_64": {"dtype": "bf16", "entries":
                       [(16, 64, 576, 1.0), (16, 128, 1152, 1.0),
                        (16, 256, 2304, 1.0), (16, 512, 4608, 1.0)]},
    # its first stage alone: 16 matrices of 64 x 576 (the fused small-matrix kernel)
    "resnet_conv_64x576_b16": {"dtype": "bf16", "entries": [(16, 64, 576, 1.0)]},
}


def workload_shapes(name: str):
    """List of (m, n, alpha, seed) for every matrix of a workload."""
    spec = WORKLOADS[name]
    out, i = [], 0
    for count, m, n, alpha in spec["entries"]:
        for _ in range(count):
            out.append((m, n, alpha, i))
            i += 1
    return out


def power_law_batch_device(count: int, m: int, n: int, alpha: float, seed: int,
                           device="cuda", dtype=None, noise: float = 0.01):
    """The same recipe drawn on the GPU with torch in float32 (benchmark inputs).

    Used where the float64 host draw of large matrices would dominate the run
    time (QR of 14336 x 4096 Gaussians); values differ from
    ``power_law_matrix`` but follow the same distribution.  Returns a
    (count, m, n) tensor cast once to ``dtype`` (default bfloat16).
    """
    import torch
    dtype = torch.bfloat16 if dtype is None else dtype
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    k = min(m, n)
    out = torch.empty((count, m, n), dtype=dtype, device=device)
    sigma = torch.arange(1, k + 1, dtype=torch.float32, device=device) ** (-float(alpha))
    for i in range(count):
        gu = torch.randn((m, k), generator=g, device=device, dtype=torch.float32)
        gv = torch.randn((n, k), generator=g, device=device, dtype=torch.float32)
        qu, ru = torch.linalg.qr(gu)
        qv, rv = torch.linalg.qr(gv)
        qu = qu * torch.sign(torch.diagonal(ru)).clamp(min=0).mul(2).sub(1)[None, :]
        qv = qv * torch.sign(torch.diagonal(rv)).clamp(min=0).mul(2).sub(1)[None, :]
        e = torch.randn((m, n), generator=g, device=device, dtype=torch.float32)
        x = (qu * sigma[None, :]) @ qv.T.contiguous() + noise * e
        out[i].copy_(x.to(dtype))
        del gu, gv, qu, qv, ru, rv, e, x
    return out

"""Fused small-matrix path (bf16 calls whose matrices all have min(m, n) <= 128
and fit in one compute unit's LDS): one launch per call, against the fp64
oracle and, bit for bit, against the tiled kernels of the same call
(TM_DISABLE_FUSED), which the rest of the GPU suite pins to the oracle."""
import contextlib
import os

import numpy as np
import pytest

from oracle import turbomuon as O
from gpu_helpers import (BF16_TOL, EO_RATIO_TOL, SCHEDULE5, eo_ratio, from_device, log,
                         make_input, relF, to_device)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402


@contextlib.contextmanager
def tiled_only():
    os.environ["TM_DISABLE_FUSED"] = "1"
    try:
        yield
    finally:
        del os.environ["TM_DISABLE_FUSED"]


def launches(fn):
    """Launch count per phase of the calls made by fn()."""
    tm.timing_reset()
    tm.timing_enable(True)
    try:
        fn()
        torch.cuda.synchronize()
    finally:
        tm.timing_enable(False)
    counts = {p: tm.timing_read(p)[1] for p in tm.PHASES}
    tm.timing_reset()
    return counts


def only_fused(counts, n=1):
    return counts["fused"] == n and all(v == 0 for p, v in counts.items() if p != "fused")


def run_batched(Xs, iters, precond, coeffs=None):
    t = torch.stack([to_device(X, "bf16") for X in Xs]).contiguous()
    tm.orthogonalize(t, iters, coeffs, precond)
    torch.cuda.synchronize()
    return t


def run_grouped(Xs, iters, precond, coeffs=None):
    ts = [to_device(X, "bf16") for X in Xs]
    tm.orthogonalize_grouped(ts, iters, coeffs, precond)
    torch.cuda.synchronize()
    return ts


PARITY = [(1, 1), (17, 33), (33, 17), (64, 576), (576, 64), (128, 320), (320, 128), (96, 96),
          (1, 128), (128, 1), (64, 1088), (100, 300)]


@pytest.mark.parametrize("m,n", PARITY)
@pytest.mark.parametrize("precond,iters", [("aol", 4), ("frobenius", 5), ("schatten4", 4)])
def test_fused_matches_oracle(m, n, precond, iters):
    log(f"case: fused {m}x{n} {precond} t={iters}")
    X = make_input(m, n, 0.8, 11 * m + n, "bf16")
    t = to_device(X, "bf16")
    counts = launches(lambda: tm.orthogonalize(t, iters, None, precond))
    assert only_fused(counts), counts
    G = from_device(t)
    R = O.orthogonalize(X, iters, None, precond)
    e = relF(G, R)
    log(f"relF={e:.3e}")
    assert e <= BF16_TOL
    if min(m, n) >= 16:
        r = eo_ratio(G, R)
        log(f"eo_ratio={r:.4f}")
        assert abs(r - 1) <= EO_RATIO_TOL


SHAPES = [(1, 1), (3, 5), (5, 3), (17, 33), (33, 17), (31, 32), (32, 31), (64, 576), (576, 64),
          (65, 129), (129, 65), (127, 200), (128, 320), (8, 1000),
          # tall with k % 8 == 0 (8 x 8 register-transposed loads and stores): a last
          # block of 8 rows only partly inside the matrix, zero columns past N
          (333, 40), (99, 8), (200, 96)]
CASES = [("aol", 4, None), ("aol", 1, None), ("frobenius", 5, None), ("schatten4", 4, None),
         ("none", 3, None), ("aol", 5, SCHEDULE5)]


@pytest.mark.parametrize("m,n", SHAPES)
@pytest.mark.parametrize("precond,iters,coeffs", CASES)
def test_fused_equals_tiled_bitwise(m, n, precond, iters, coeffs):
    log(f"case: fused vs tiled 3 x {m}x{n} {precond} t={iters}")
    Xs = [make_input(m, n, 1.0, 100 * b + m + 3 * n, "bf16") for b in range(3)]
    if precond == "none":
        Xs = [X / max(np.linalg.norm(X, 2), 1e-30) for X in Xs]
        Xs = [to_device(X, "bf16").float().cpu().numpy().astype(np.float64) for X in Xs]
    f = run_batched(Xs, iters, precond, coeffs)
    with tiled_only():
        g = run_batched(Xs, iters, precond, coeffs)
    assert torch.equal(f.view(torch.int16), g.view(torch.int16))
    assert torch.isfinite(f.float()).all()


def test_grouped_many_shapes_several_launches_bitwise():
    """More entries and table pointers than one launch holds (32 / 64): the
    call is split into several launches per class; every matrix equals the
    tiled kernels' result and its own single call, bit for bit."""
    rng = np.random.default_rng(5)
    shapes = []
    for i in range(150):
        k = int(rng.integers(1, 129))
        N = int(rng.integers(k, 321))
        shapes.append((k, N) if i % 3 else (N, k))
    shapes += [(64, 576)] * 70          # one long run of a shape: pointer table split
    log(f"case: grouped {len(shapes)} small matrices")
    Xs = [make_input(m, n, 1.0, 1000 + i, "bf16") for i, (m, n) in enumerate(shapes)]
    holder = {}
    counts = launches(lambda: holder.setdefault("f", run_grouped(Xs, 4, "aol")))
    assert counts["fused"] >= 4 and all(v == 0 for p, v in counts.items() if p != "fused"), counts
    f = holder["f"]
    with tiled_only():
        g = run_grouped(Xs, 4, "aol")
    for i in range(len(Xs)):
        assert torch.equal(f[i].view(torch.int16), g[i].view(torch.int16)), shapes[i]
    for i in (0, 1, 2, 77, 149, 160, 219):
        s = run_batched([Xs[i]], 4, "aol")[0]
        assert torch.equal(s.view(torch.int16), f[i].view(torch.int16)), shapes[i]
    for i in (0, 1, 2, 160):
        e = relF(from_device(f[i]), O.orthogonalize(Xs[i], 4, None, "aol"))
        log(f"{shapes[i]} relF={e:.3e}")
        assert e <= BF16_TOL


def test_conv_stage_16x64x576_one_launch_deterministic():
    """16 matrices of 64 x 576: one launch, the same bits on every call, batched
    equals grouped."""
    Xs = [make_input(64, 576, 1.0, 300 + i, "bf16") for i in range(16)]
    t = torch.stack([to_device(X, "bf16") for X in Xs]).contiguous()
    first = t.clone()
    counts = launches(lambda: tm.orthogonalize(first, 4, None, "aol"))
    assert only_fused(counts), counts
    for _ in range(3):
        again = t.clone()
        tm.orthogonalize(again, 4, None, "aol")
        torch.cuda.synchronize()
        assert torch.equal(again.view(torch.int16), first.view(torch.int16))
    gs = run_grouped(Xs, 4, "aol")
    for i in range(16):
        assert torch.equal(gs[i].view(torch.int16), first[i].view(torch.int16))
    e = relF(from_device(first[5]), O.orthogonalize(Xs[5], 4, None, "aol"))
    assert e <= BF16_TOL


def test_mixed_call_stays_tiled():
    """A call with one matrix too large for the LDS runs every matrix on the
    tiled kernels: no fused launch."""
    Xs = [make_input(64, 576, 1.0, 1, "bf16"), make_input(256, 512, 1.0, 2, "bf16")]
    holder = {}
    counts = launches(lambda: holder.setdefault("f", run_grouped(Xs, 4, "aol")))
    assert counts["fused"] == 0 and counts["update"] > 0, counts
    single = run_batched([Xs[0]], 4, "aol")[0]
    assert torch.equal(single.view(torch.int16), holder["f"][0].view(torch.int16))


def test_fused_iters0_and_f32_are_not_fused():
    X = make_input(40, 70, 1.0, 4, "bf16")
    t = to_device(X, "bf16")
    counts = launches(lambda: tm.orthogonalize(t, 0, None, "aol"))
    assert counts["fused"] == 0
    assert relF(from_device(t), O.preconditioned(X, "aol")) <= 4e-3
    u = to_device(X, "f32")
    counts = launches(lambda: tm.orthogonalize(u, 4, None, "aol"))
    assert counts["fused"] == 0


def test_fused_unaligned_rows_and_odd_pointers():
    """Rows of odd length and a matrix starting 2 bytes past a 16-byte boundary
    take the element-wise edges of the loads and stores."""
    for m, n in ((7, 13), (13, 7), (64, 577), (577, 64)):
        X = make_input(m, n, 1.0, m + n, "bf16")
        buf = torch.zeros(m * n + 1, dtype=torch.bfloat16, device="cuda")
        view = buf[1:].view(m, n)
        view.copy_(to_device(X, "bf16"))
        tm.orthogonalize(view, 4, None, "aol")
        ref = run_batched([X], 4, "aol")[0]
        with tiled_only():
            til = run_batched([X], 4, "aol")[0]
        torch.cuda.synchronize()
        assert buf[0].item() == 0.0
        assert torch.equal(view.view(torch.int16), til.view(torch.int16)), (m, n)
        assert torch.equal(ref.view(torch.int16), til.view(torch.int16)), (m, n)


def test_noalloc_small_call_is_fused():
    Xs = [make_input(96, 300, 1.0, 60 + i, "bf16") for i in range(4)]
    a = torch.stack([to_device(X, "bf16") for X in Xs]).contiguous()
    b = a.clone()
    counts = launches(lambda: tm.orthogonalize(b, 4, None, "aol"))
    assert only_fused(counts)
    tm.orthogonalize_noalloc(a, 4, None, "aol")
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_fused_every_iteration_row_of_the_descriptor():
    """TM_MAX_ITERS iterations: every coefficient row the launch descriptor holds is
    used (a normalised quintic schedule cycled to 64 rows), bitwise equal to the
    tiled kernels."""
    rows = [SCHEDULE5[i % 5] for i in range(tm.TM_MAX_ITERS)]
    Xs = [make_input(40, 200, 1.0, 77 + b, "bf16") for b in range(2)]
    f = run_batched(Xs, tm.TM_MAX_ITERS, "aol", rows)
    with tiled_only():
        g = run_batched(Xs, tm.TM_MAX_ITERS, "aol", rows)
    assert torch.equal(f.view(torch.int16), g.view(torch.int16))
    e = relF(from_device(f[0]), O.orthogonalize(Xs[0], tm.TM_MAX_ITERS, rows, "aol"))
    log(f"t=64 relF={e:.3e}")
    assert e <= BF16_TOL


@pytest.mark.parametrize("seed", range(4))
def test_fused_random_shapes_equal_tiled(seed):
    """Seeded random shapes across the fused kernel's range (k <= 128, both LDS
    variants, both orientations) and pre-conditionings: bitwise the tiled kernels."""
    rng = np.random.default_rng(900 + seed)
    shapes = []
    while len(shapes) < 6:
        k = int(rng.integers(1, 129))
        N = int(rng.integers(k, 1200))
        m, n = (k, N) if rng.integers(2) else (N, k)
        kp, Np = -(-k // 32) * 32, -(-N // 32) * 32
        lds = kp * (2 * Np + 16) + 2 * kp * (2 * kp + 16) + (kp // 16) * kp * 4 + kp * 4 + 512
        if lds <= 160 * 1024:
            shapes.append((m, n))
    precond = ("aol", "frobenius", "schatten4", "aol")[seed]
    iters = (4, 5, 4, 2)[seed]
    log(f"case: random fused shapes {shapes} {precond} t={iters}")
    Xs = [make_input(m, n, 0.9, 1000 * seed + i, "bf16") for i, (m, n) in enumerate(shapes)]
    counts = launches(lambda: run_grouped(Xs, iters, precond))
    # one launch per (kp / 32, LDS variant) class present in the group
    assert counts["fused"] >= 1 and all(v == 0 for p, v in counts.items() if p != "fused"), counts
    f = run_grouped(Xs, iters, precond)
    with tiled_only():
        g = run_grouped(Xs, iters, precond)
    for i in range(len(shapes)):
        assert torch.equal(f[i].view(torch.int16), g[i].view(torch.int16)), shapes[i]


def test_fused_large_batch_of_tiny_matrices():
    """65 537 matrices of 3 x 5 in one batched call: one workgroup each in one
    launch, bitwise the tiled kernels."""
    g = torch.Generator(device="cuda")
    g.manual_seed(5)
    X = torch.randn((65537, 3, 5), generator=g, device="cuda").bfloat16()
    f = X.clone()
    counts = launches(lambda: tm.orthogonalize(f, 4, None, "aol"))
    assert only_fused(counts), counts
    t = X.clone()
    with tiled_only():
        tm.orthogonalize(t, 4, None, "aol")
        torch.cuda.synchronize()
    assert torch.equal(f.view(torch.int16), t.view(torch.int16))
    e = relF(from_device(f[65536]), O.orthogonalize(from_device(X[65536]), 4, None, "aol"))
    assert e <= BF16_TOL

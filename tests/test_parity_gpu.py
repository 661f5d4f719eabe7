"""Parity of the HIP path (through the C ABI) with the fp64 oracle."""
import numpy as np
import pytest

from oracle import turbomuon as O
from paper_2512_04632_amd import synth
from gpu_helpers import (BF16_TOL, F32_TOL, EO_RATIO_TOL, SCHEDULE5, block_relF_max, from_device,
                         log, make_input, normalised_quintic, relF, eo_ratio, to_device)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2512_04632_amd import _lib as tm  # noqa: E402


def gpu_orth(Xc, dtype, iters, precond, coeffs=None):
    t = to_device(Xc, dtype)
    tm.orthogonalize(t, iters, coeffs, precond)
    torch.cuda.synchronize()
    return from_device(t)


def tol(dtype):
    return BF16_TOL if dtype == "bf16" else F32_TOL


# ----------------------------------------------------------------- single matrices
def test_single_256_fp32_aol4():
    log("case: 256x256 fp32 alpha=1 seed=0 AOL t=4")
    X = make_input(256, 256, 1.0, 0, "f32")
    G = gpu_orth(X, "f32", 4, "aol")
    R = O.orthogonalize(X, 4, None, "aol")
    e = relF(G, R)
    Q = O.polar_factor(X)
    pg, po = O.eps_polar(G, X, Q), O.eps_polar(R, X, Q)
    log(f"relF={e:.3e} eps_polar gpu={pg:.4f} oracle={po:.4f}")
    assert e <= F32_TOL
    assert abs(pg - po) <= 0.05 * po   # distance to the SVD polar factor (Section 3)


@pytest.mark.parametrize("precond,iters", [("aol", 4), ("frobenius", 5)])
def test_gpt2_mlp_768x3072_bf16(precond, iters):
    log(f"case: 768x3072 bf16 alpha=0.8 seed=0 {precond} t={iters}")
    X = make_input(768, 3072, 0.8, 0, "bf16")
    G = gpu_orth(X, "bf16", iters, precond)
    R = O.orthogonalize(X, iters, None, precond)
    e, r = relF(G, R), eo_ratio(G, R)
    log(f"relF={e:.3e} eo_ratio={r:.4f}")
    assert e <= BF16_TOL
    assert abs(r - 1) <= EO_RATIO_TOL


SHAPES = [(1, 1), (1, 8), (8, 1), (5, 3), (17, 33), (33, 17), (64, 64), (100, 300), (300, 100),
          (129, 130), (64, 576), (257, 520), (520, 257), (96, 1000)]


@pytest.mark.parametrize("m,n", SHAPES)
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("precond,iters", [("aol", 4), ("frobenius", 5), ("aol", 1),
                                           ("schatten4", 4)])
def test_shapes(m, n, dtype, precond, iters):
    log(f"case: {m}x{n} {dtype} {precond} t={iters}")
    X = make_input(m, n, 0.8, m * 7 + n, dtype)
    G = gpu_orth(X, dtype, iters, precond)
    R = O.orthogonalize(X, iters, None, precond)
    e = relF(G, R)
    log(f"relF={e:.3e}")
    assert e <= tol(dtype)


# 3 x 40000 bf16 with Frobenius scaling and 5 iterations misses the bf16
# tolerance whatever the kernels do: a NumPy model of the bf16 storage points
# (one rounding per stored X, A, B) gives 3.11e-2 on this input, like the GPU.
# With k = 3 the constant triple's steep slope near the normalised singular
# values amplifies the rounding of X over five iterations; over 12 seeds the
# model exceeds 2e-2 on 6 (median 1.7e-2), and adding a X in the fp32 epilogue
# instead of folding a into the stored polynomial changes the seeds that fail,
# not their number (5 of 12).  AOL (4.8e-3) and Schatten-4 (8.5e-3) meet it.
_BF16_K3_FROB = pytest.mark.xfail(strict=True, reason=(
    "bf16 storage error amplified past 2e-2 at k = 3, Frobenius, t = 5 (3.1e-2 in the "
    "rounding model of the same input)"))


def _extreme_cases():
    out = []
    for m, n in [(1, 65536), (65536, 1), (3, 40000), (40000, 3)]:
        for dtype, precond, iters in [("bf16", "aol", 4), ("bf16", "frobenius", 5),
                                      ("bf16", "schatten4", 4), ("f32", "aol", 4),
                                      ("f32", "frobenius", 5), ("f32", "schatten4", 4)]:
            marks = (_BF16_K3_FROB,) if (m, n, dtype, precond) == (3, 40000, "bf16",
                                                                   "frobenius") else ()
            out.append(pytest.param(m, n, dtype, precond, iters, marks=marks))
    return out


@pytest.mark.parametrize("m,n,dtype,precond,iters", _extreme_cases())
def test_extreme_aspect_ratios(m, n, dtype, precond, iters):
    """One side at or near the largest dimension, the other tiny."""
    log(f"case: {m}x{n} {dtype} {precond} t={iters}")
    X = make_input(m, n, 0.8, m * 7 + n, dtype)
    G = gpu_orth(X, dtype, iters, precond)
    R = O.orthogonalize(X, iters, None, precond)
    e = relF(G, R)
    log(f"relF={e:.3e}")
    assert e <= tol(dtype)


@pytest.mark.parametrize("m,n", [(17, 33), (33, 17), (256, 256), (100, 300), (300, 100)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("precond", ["aol", "frobenius", "schatten4"])
def test_iters0_is_preconditioned_input(m, n, dtype, precond):
    log(f"case: iters=0 {m}x{n} {dtype} {precond}")
    X = make_input(m, n, 1.0, 3, dtype)
    G = gpu_orth(X, dtype, 0, precond)
    R = O.preconditioned(X, precond)
    assert relF(G, R) <= (4e-3 if dtype == "bf16" else 1e-6)
    u = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -24
    assert np.linalg.norm(G, 2) <= 1 + 4 * u   # AOL / Frobenius / Schatten-4 bound ||X1||_2 <= 1


def test_precond_none_and_iters0_none_is_identity():
    X = make_input(40, 70, 1.0, 1, "bf16")
    X = synth.cast(X / np.linalg.norm(X, 2), "bf16")
    assert np.array_equal(gpu_orth(X, "bf16", 0, "none"), X)
    G = gpu_orth(X, "bf16", 3, "none")
    assert relF(G, O.orthogonalize(X, 3, None, "none")) <= BF16_TOL


# Coefficient choices that isolate the steps: (1,0,0) keeps X1, (0,1,0) gives
# X1 X1^T X1 (Gram + update), (0,0,1) gives (X1 X1^T)^2 X1 (Gram, poly, update).
@pytest.mark.parametrize("coeffs", [[(1.0, 0.0, 0.0)], [(0.0, 1.0, 0.0)], [(0.0, 0.0, 1.0)],
                                    [(1.5, -0.5, 0.0)] * 3,
                                    [normalised_quintic(a) for a in (3.2, 2.5, 2.0, 1.7)]])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("m,n", [(130, 250), (250, 130)])
def test_step_isolating_coefficients(coeffs, dtype, m, n):
    log(f"case: coeffs={coeffs[0]}.. {m}x{n} {dtype}")
    X = make_input(m, n, 0.8, 5, dtype)
    G = gpu_orth(X, dtype, len(coeffs), "aol", coeffs)
    R = O.orthogonalize(X, len(coeffs), coeffs, "aol")
    assert relF(G, R) <= tol(dtype)


@pytest.mark.parametrize("t", [4, 2])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("m,n", [(200, 520), (520, 200)])
def test_truncated_schedule_runs_the_last_rows(t, dtype, m, n):
    """Appendix on the tuning of Newton-Schulz coefficients: t iterations from a
    five-row schedule run its last t rows (tm_schedule_tail), e.g. rows 2..5 for
    t = 4.  Where the oracle's results for the last and the first t rows are far
    enough apart for the tolerance to tell them apart, the GPU result must also be
    far from the first rows' (fp64: 8e-3 apart at t = 4, 0.6 at t = 2)."""
    log(f"case: last {t} rows of a 5-row schedule, {m}x{n} {dtype}")
    rows = tm.schedule_tail(SCHEDULE5, t)
    X = make_input(m, n, 0.8, 21, dtype)
    G = gpu_orth(X, dtype, t, "aol", rows)
    R = O.orthogonalize(X, t, O.schedule_last(SCHEDULE5, t), "aol")
    e = relF(G, R)
    log(f"relF={e:.3e}")
    assert e <= tol(dtype)
    W = O.orthogonalize(X, t, SCHEDULE5[:t], "aol")
    if relF(W, R) > 20 * tol(dtype):
        assert relF(G, W) > 10 * tol(dtype)


def test_zero_matrix_and_zero_row():
    for dtype in ("bf16", "f32"):
        for pre in ("aol", "frobenius", "schatten4"):
            Z = np.zeros((48, 80))
            assert np.all(gpu_orth(Z, dtype, 4, pre) == 0)
        X = make_input(48, 80, 1.0, 2, dtype)
        X[7] = 0.0
        G = gpu_orth(X, dtype, 4, "aol")
        assert np.all(G[7] == 0) and np.all(np.isfinite(G))
        assert relF(G, O.orthogonalize(X, 4)) <= tol(dtype)


# ----------------------------------------------------------------- batch / group equality
@pytest.mark.parametrize("m,n", [(96, 200), (200, 96), (256, 256)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_batched_grouped_single_are_bitwise_equal(m, n, dtype):
    log(f"case: batch/group equality {m}x{n} {dtype}")
    Xs = [make_input(m, n, 0.8, s, dtype) for s in range(3)]
    single = [gpu_orth(X, dtype, 4, "aol") for X in Xs]
    tb = torch.stack([to_device(X, dtype) for X in Xs]).contiguous()
    tm.orthogonalize(tb, 4, None, "aol")
    tg = [to_device(X, dtype) for X in Xs]
    tm.orthogonalize_grouped(tg, 4, None, "aol")
    torch.cuda.synchronize()
    for i in range(3):
        assert np.array_equal(from_device(tb[i]), single[i])
        assert np.array_equal(from_device(tg[i]), single[i])
    again = gpu_orth(Xs[0], dtype, 4, "aol")
    assert np.array_equal(again, single[0])        # run-to-run determinism


# ----------------------------------------------------------------- one-stage main loops
@pytest.mark.parametrize("m,n", [(64, 64), (40, 56)])
def test_many_small_matrices_one_stage_loops(m, n):
    """300 matrices padded to 64 x 64: the batched call's first Gram and its updates
    run more than 256 tiles of 64, so their ring stages are 64 wide and K = 64 is a
    single stage (the producer-wave loop and the update loop with one stage); the
    grouped call splits them over launches of at most 96 matrices (the pointer table
    of one launch), with other stage widths.
    Both must agree bit for bit with single calls and stay within the oracle's
    tolerance."""
    log(f"case: batch of 300 {m}x{n} bf16 AOL t=4")
    Xs = [make_input(m, n, 0.8, 1000 + s, "bf16") for s in range(300)]
    tb = torch.stack([to_device(X, "bf16") for X in Xs]).contiguous()
    tm.orthogonalize(tb, 4, None, "aol")
    tg = [to_device(X, "bf16") for X in Xs]
    tm.orthogonalize_grouped(tg, 4, None, "aol")
    torch.cuda.synchronize()
    for i in range(0, 300, 37):
        G = from_device(tb[i])
        assert np.array_equal(from_device(tg[i]), G), i
        assert np.array_equal(gpu_orth(Xs[i], "bf16", 4, "aol"), G), i
        assert relF(G, O.orthogonalize(Xs[i], 4)) <= BF16_TOL, i


def test_grouped_entry_and_pointer_limits():
    """A grouped call whose matrices need more launch entries (runs of one shape share
    an entry through the pointer table, other matrices take one entry each) and more
    table pointers than one launch holds: 12 blocks of a run of three 32 x 48 matrices
    and seven single matrices of other shapes (96 entries), then a run of 100 64 x 64
    matrices.  Every matrix must equal its single call bit for bit."""
    log("case: grouped call over the entry and pointer-table limits")
    block = [(32, 48)] * 3 + [(24, 40), (40, 24), (17, 33), (33, 17), (20, 20), (48, 32), (5, 9)]
    shapes = block * 12 + [(64, 64)] * 100
    Xs = [make_input(m, n, 0.8, 5000 + i, "bf16") for i, (m, n) in enumerate(shapes)]
    ts = [to_device(X, "bf16") for X in Xs]
    tm.orthogonalize_grouped(ts, 4, None, "aol")
    torch.cuda.synchronize()
    for i in list(range(0, 120, 7)) + [120, 150, 215, 216, 219]:
        G = from_device(ts[i])
        assert np.array_equal(G, gpu_orth(Xs[i], "bf16", 4, "aol")), i
    for i in (0, 3, 219):
        assert relF(from_device(ts[i]), O.orthogonalize(Xs[i], 4)) <= BF16_TOL, i


def test_fused_aol_vector_matches_separate_launch_bitwise():
    """With k <= 1024 the rescale pass sums the AOL vector itself; a call that also
    holds a matrix with k > 1024 takes the separate AOL-vector launch for all of its
    matrices.  Both add the same row partials in the same order: equal bits."""
    log("case: fused vs separate AOL vector, bitwise")
    Xs = [make_input(1100, 1200, 0.8, 71, "bf16"), make_input(300, 700, 0.8, 72, "bf16"),
          make_input(1024, 1030, 0.8, 73, "bf16")]
    ts = [to_device(X, "bf16") for X in Xs]
    tm.orthogonalize_grouped(ts, 4, None, "aol")
    torch.cuda.synchronize()
    for i, X in enumerate(Xs):
        G = from_device(ts[i])
        assert np.array_equal(G, gpu_orth(X, "bf16", 4, "aol")), i
        assert relF(G, O.orthogonalize(X, 4)) <= BF16_TOL, i


# ----------------------------------------------------------------- grouped workloads
def run_workload(name, iters=4, precond="aol"):
    shapes = synth.workload_shapes(name)
    dtype = synth.WORKLOADS[name]["dtype"]
    Xs = [make_input(m, n, a, s, dtype) for (m, n, a, s) in shapes]
    ts = [to_device(X, dtype) for X in Xs]
    tm.orthogonalize_grouped(ts, iters, None, precond)
    torch.cuda.synchronize()
    return Xs, [from_device(t) for t in ts]


def _check_group(Xs, Gs):
    """Every matrix of a grouped call against the oracle: global and per 256 x 256
    block relative error, and the polar-error ratio."""
    worst, worst_b = 0.0, 0.0
    for i, (X, G) in enumerate(zip(Xs, Gs)):
        R = O.orthogonalize(X, 4)
        e, r, eb = relF(G, R), eo_ratio(G, R), block_relF_max(G, R)
        worst, worst_b = max(worst, e), max(worst_b, eb)
        assert e <= BF16_TOL and eb <= BF16_TOL and abs(r - 1) <= EO_RATIO_TOL, (i, e, eb, r)
    log(f"{len(Xs)} matrices: worst relF={worst:.3e}, worst 256-block relF={worst_b:.3e}")


def test_grouped_gpt2_small_72_matrices():
    log("case: grouped gpt2_small_12layer (72 matrices)")
    Xs, Gs = run_workload("gpt2_small_12layer")
    _check_group(Xs, Gs)


def test_grouped_gpt2_small_matches_single_calls_bitwise():
    """The grouped call runs 256-tiles (after the sort by product size its last 16
    update tiles belong to the last two 768 x 768 matrices, 46 and 47, and run as
    4 x 4 sub-tiles of 64 x 64); a single 3072 x 768 call runs 64-tiles.  Every
    output element sees the same products in the same order: equal bits."""
    log("case: grouped gpt2_small_12layer vs single calls, bitwise")
    shapes = synth.workload_shapes("gpt2_small_12layer")
    Xs = [make_input(m, n, a, s, "bf16") for (m, n, a, s) in shapes]
    ts = [to_device(X, "bf16") for X in Xs]
    tm.orthogonalize_grouped(ts, 4, None, "aol")
    for i in (0, 45, 46, 47, 48, 59, 60, 71):
        assert torch.equal(ts[i], (lambda t: (tm.orthogonalize(t, 4, None, "aol"), t)[1])(
            to_device(Xs[i], "bf16"))), i
    torch.cuda.synchronize()


def test_grouped_mixed_k_dealt_by_matrix_matches_single_calls():
    """A grouped launch whose Gram tiles differ in K, and whose matrices split
    evenly over the 8 XCDs, deals whole matrices round-robin to the XCDs: 24
    matrices of 256 x 2048 and 30 of 256 x 512 (540 Gram tiles of 64; queues of 70
    and 60 tiles per XCD, so some workgroups find no tile).  Every matrix equals
    its own single call bit for bit, and a sample of each shape the oracle."""
    log("case: grouped 24 x 256x2048 + 30 x 256x512, by-matrix dealing")
    shapes = [(256, 2048)] * 24 + [(256, 512)] * 30
    Xs = [make_input(m, n, 0.8, 500 + i, "bf16") for i, (m, n) in enumerate(shapes)]
    ts = [to_device(X, "bf16") for X in Xs]
    tm.orthogonalize_grouped(ts, 4, None, "aol")
    torch.cuda.synchronize()
    for i in range(len(shapes)):
        single = to_device(Xs[i], "bf16")
        tm.orthogonalize(single, 4, None, "aol")
        assert torch.equal(ts[i], single), i
    for i in (0, 23, 24, 53):
        e = relF(from_device(ts[i]), O.orthogonalize(Xs[i], 4, None, "aol"))
        log(f"matrix {i}: relF={e:.3e}")
        assert e <= BF16_TOL


@pytest.mark.parametrize("precond", ["schatten4", "aol", "frobenius"])
def test_small_matrix_alone_and_beside_large_ones_bitwise(precond):
    """A 100 x 300 matrix alone (fused kernel) and in a group with two 2048 x 8192
    matrices (tiled kernels on 256 x 256 tiles, its rows padded to 256): the same
    bits.  The Schatten-4 sums are chunked by the 64-column partials of the k real
    rows, not of the padded width, so the tile size does not enter them."""
    log(f"case: 100x300 alone vs beside 2 x 2048x8192, {precond}")
    small = make_input(100, 300, 0.8, 41, "bf16")
    big = [make_input(2048, 8192, 0.5, 42 + i, "bf16") for i in range(2)]
    alone = to_device(small, "bf16")
    tm.orthogonalize(alone, 4, None, precond)
    ts = [to_device(small, "bf16")] + [to_device(b, "bf16") for b in big]
    tm.orthogonalize_grouped(ts, 4, None, precond)
    torch.cuda.synchronize()
    assert torch.equal(alone, ts[0])
    e = relF(from_device(ts[0]), O.orthogonalize(small, 4, None, precond))
    assert e <= BF16_TOL


def test_grouped_resnet_conv_64_matrices():
    log("case: grouped resnet_conv_64 (64 matrices)")
    Xs, Gs = run_workload("resnet_conv_64")
    _check_group(Xs, Gs)


@pytest.mark.parametrize("m,n", [(768, 3072), (3072, 768)])
def test_schatten4_gpt2_mlp_bf16(m, n):
    log(f"case: {m}x{n} bf16 alpha=0.8 seed=0 schatten4 t=4")
    X = make_input(m, n, 0.8, 0, "bf16")
    G = gpu_orth(X, "bf16", 4, "schatten4")
    R = O.orthogonalize(X, 4, None, "schatten4")
    e, r = relF(G, R), eo_ratio(G, R)
    log(f"relF={e:.3e} eo_ratio={r:.4f}")
    assert e <= BF16_TOL
    assert abs(r - 1) <= EO_RATIO_TOL


@pytest.mark.parametrize("m,n", [(256, 512), (768, 3072)])
@pytest.mark.parametrize("precond,iters", [("aol", 4), ("frobenius", 5), ("schatten4", 2),
                                           ("none", 3), ("aol", 0), ("aol", 1)])
def test_in_place_first_iteration_matches_padded_copy(m, n, precond, iters):
    """A wide matrix whose dims are multiples of the tile is read in place by the
    first iteration when 16-byte aligned; one stored 2 bytes past an alignment
    boundary goes through the padded copy.  Same arithmetic, same bits."""
    log(f"case: in-place vs copied first iteration {m}x{n} {precond} t={iters}")
    X = make_input(m, n, 0.8, 9, "bf16")
    a = to_device(X, "bf16")
    buf = torch.empty(m * n + 8, dtype=torch.bfloat16, device="cuda")
    b = buf[1:1 + m * n].view(m, n)
    b.copy_(a)
    assert a.data_ptr() % 16 == 0 and b.data_ptr() % 16 == 2
    tm.orthogonalize(a, iters, None, precond)
    tm.orthogonalize(b, iters, None, precond)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    R = O.orthogonalize(X, iters, None, precond)
    assert relF(from_device(a), R) <= (4e-3 if iters == 0 else BF16_TOL)

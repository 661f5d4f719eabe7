"""Pins of the fp64 oracle against facts fixed by the paper and by linear algebra.

None of these re-types the oracle's own loop: each compares it with an
independent route (SVD closed forms, limits, hand-derived special cases,
bounds, invariances, a printed value).
"""
import json
import os

import numpy as np
import pytest

from oracle import turbomuon as O
from paper_2512_04632_amd import synth
from gpu_helpers import SCHEDULE5

TRIPLE = O.CONSTANT_TRIPLE
HERE = os.path.dirname(os.path.abspath(__file__))


def phi(x, coeffs):
    """Scalar composition p_t o ... o p_1, p(x) = a x + b x^3 + c x^5.

    An odd matrix polynomial of eq. (ns_quintic) acts on each singular value
    separately, so this scalar map fixes the whole iteration's output.
    """
    x = np.asarray(x, dtype=np.float64)
    for a, b, c in coeffs:
        x = a * x + b * x ** 3 + c * x ** 5
    return x


def spectral_closed_form(X1, coeffs):
    U, sv, Vt = np.linalg.svd(X1, full_matrices=False)
    return (U * phi(sv, coeffs)[None, :]) @ Vt


def relF(a, b):
    return np.linalg.norm(a - b) / np.linalg.norm(b)


def rand_orth(rng, n):
    q, r = np.linalg.qr(rng.standard_normal((n, n)))
    return q * np.sign(np.diag(r))[None, :]


# --------------------------------------------------------------------------
# P1: the loop equals U phi(Sigma) V^T (textbook SVD + scalar polynomial)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("m,n", [(17, 33), (40, 40), (64, 20), (1, 7), (7, 1), (96, 96)])
@pytest.mark.parametrize("precond", ["aol", "frobenius", "schatten4", "none"])
def test_p1_loop_matches_spectral_closed_form(m, n, precond):
    rng = np.random.default_rng(m * 1000 + n)
    X = synth.power_law_matrix(m, n, 0.8, seed=m + n)
    if precond == "none":
        X = X * (1.1 / np.linalg.norm(X, 2))
    X1 = O.preconditioned(X, precond)
    for t, coeffs in [(4, [TRIPLE] * 4), (5, [TRIPLE] * 5),
                      (3, [tuple(rng.uniform([1.5, -2.5, 0.2], [3.5, -1.0, 1.0])) for _ in range(3)])]:
        Z = O.orthogonalize(X, t, coeffs, precond)
        assert relF(Z, spectral_closed_form(X1, coeffs)) <= 1e-11


def test_p1_each_step_is_the_direct_quintic():
    """Alg. 1's three steps equal eq. (ns_quintic)'s direct form, brute force in loops."""
    X = synth.power_law_matrix(3, 5, 1.0, seed=3)
    X1 = O.preconditioned(X, "none") * 0.5
    a, b, c = TRIPLE
    m, n = X1.shape

    def mm(P, Q):
        return [[sum(P[i][l] * Q[l][j] for l in range(len(Q))) for j in range(len(Q[0]))]
                for i in range(len(P))]

    def tr(P):
        return [list(r) for r in zip(*P)]

    x = X1.tolist()
    xxt = mm(x, tr(x))
    x3 = mm(xxt, x)                      # X X^T X
    x5 = mm(xxt, x3)                     # X X^T X X^T X
    direct = np.array([[a * x[i][j] + b * x3[i][j] + c * x5[i][j] for j in range(n)]
                       for i in range(m)])
    Z = O.orthogonalize(X1, 1, None, "none")
    assert np.max(np.abs(Z - direct)) <= 1e-14
    Zc = O.orthogonalize(X1, 1, None, "none", side="cols")  # the odd polynomial is side-free
    assert np.max(np.abs(Zc - direct)) <= 1e-14


# --------------------------------------------------------------------------
# AOL of eq. (aol), written out element by element
# --------------------------------------------------------------------------
@pytest.mark.parametrize("m,n", [(5, 3), (3, 5), (4, 4)])
def test_aol_brute_force_eq_aol(m, n):
    X = synth.power_law_matrix(m, n, 0.5, seed=11)
    # eq. (aol): column j of X0 is divided by sqrt(sum_i |(X0^T X0)_{j i}|)
    def aol_cols(P):
        p, q = len(P), len(P[0])
        g = [[sum(P[r][i] * P[r][j] for r in range(p)) for j in range(q)] for i in range(q)]
        d = [sum(abs(g[j][i]) for i in range(q)) ** -0.5 for j in range(q)]
        return np.array([[P[r][j] * d[j] for j in range(q)] for r in range(p)])

    cols = aol_cols(X.tolist())
    rows = aol_cols(X.T.tolist()).T
    assert np.max(np.abs(O.preconditioned(X, "aol", side="cols") - cols)) <= 1e-14
    assert np.max(np.abs(O.preconditioned(X, "aol", side="rows") - rows)) <= 1e-14
    auto = rows if m <= n else cols
    assert np.max(np.abs(O.preconditioned(X, "aol") - auto)) <= 1e-14
    assert np.max(np.abs(O.aol(X) - cols)) <= 1e-14


# --------------------------------------------------------------------------
# Hand-derived special cases
# --------------------------------------------------------------------------
def test_diagonal_input_is_phi1_times_sign():
    d = np.array([3.0, -0.5, 2e-3, 7.0, -1.0])
    X = np.diag(d)
    for t in (1, 4, 5):
        Z = O.orthogonalize(X, t)
        assert np.max(np.abs(Z - phi(1.0, [TRIPLE] * t) * np.diag(np.sign(d)))) <= 1e-14


def test_rank_one_is_exact_after_aol():
    """X = u v^T: the AOL scaling makes X1 = w v^T/|v| with |w| = 1 (derived by hand)."""
    rng = np.random.default_rng(5)
    u, v = rng.standard_normal(6), rng.standard_normal(9)
    X = np.outer(u, v)                               # wide: rows are scaled
    w = np.sign(u) * np.sqrt(np.abs(u) / np.abs(u).sum())
    X1 = np.outer(w, v / np.linalg.norm(v))
    assert np.max(np.abs(O.preconditioned(X, "aol") - X1)) <= 1e-14
    for t in (1, 4):
        assert np.max(np.abs(O.orthogonalize(X, t) - phi(1.0, [TRIPLE] * t) * X1)) <= 1e-13


def test_scaled_orthogonal_rows_and_columns_are_restored():
    """AOL is exact on matrices with orthogonal rows (wide) or columns (tall)."""
    rng = np.random.default_rng(7)
    Q = rand_orth(rng, 12)[:5]                       # 5 x 12, orthonormal rows
    D = np.array([4.0, -0.1, 2.0, 9.0, -3.0])
    assert np.max(np.abs(O.preconditioned(D[:, None] * Q, "aol") - np.sign(D)[:, None] * Q)) <= 1e-14
    T = Q.T * D[None, :]                             # 12 x 5, orthogonal columns
    assert np.max(np.abs(O.preconditioned(T, "aol") - Q.T * np.sign(D)[None, :])) <= 1e-14


def test_zero_matrix_and_zero_rows():
    Z = np.zeros((4, 6))
    for pre in ("aol", "frobenius", "schatten4", "none"):
        assert np.all(O.orthogonalize(Z, 4, None, pre) == 0)
    X = synth.power_law_matrix(5, 8, 1.0, seed=1)
    X[2] = 0.0
    out = O.orthogonalize(X, 4)
    assert np.all(out[2] == 0) and np.all(np.isfinite(out))
    assert np.all(O.aol_vector(X @ X.T)[2] == 0)


# --------------------------------------------------------------------------
# P2: limits -> SVD polar factors
# --------------------------------------------------------------------------
CONVERGENT = {"quintic": (15 / 8, -10 / 8, 3 / 8), "bjorck": (1.5, -0.5, 0.0)}


@pytest.mark.parametrize("kind", sorted(CONVERGENT))
@pytest.mark.parametrize("m,n", [(48, 96), (96, 48), (64, 64)])
def test_p2_converges_to_polar_of_aol_input(kind, m, n):
    X = synth.gaussian_matrix(m, n, seed=m + 2 * n)
    t = 60
    Z = O.orthogonalize(X, t, [CONVERGENT[kind]] * t, "aol")
    Qa = O.polar_factor(O.preconditioned(X, "aol"))
    assert relF(Z, Qa) <= 1e-12
    # the limit is PolarFactor(AOL(X)), not PolarFactor(X), for a generic input
    assert O.eps_bias(X) > 1e-3
    assert O.eps_approx(Z, X) <= 1e-12


def test_p2_orthogonal_rows_limit_is_polar_of_x():
    rng = np.random.default_rng(9)
    Q = rand_orth(rng, 40)[:16]
    X = np.linspace(0.2, 5.0, 16)[:, None] * Q
    t = 30
    Z = O.orthogonalize(X, t, [CONVERGENT["quintic"]] * t, "aol")
    assert relF(Z, O.polar_factor(X)) <= 1e-12
    assert O.eps_bias(X) <= 1e-13


# --------------------------------------------------------------------------
# P3: the AOL bound ||X1||_2 <= 1 (Section 4.1; Gershgorin argument of Section 5)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("m,n,alpha", [(64, 576, 1.0), (256, 256, 1.0), (200, 90, 0.5), (33, 17, 0.0)])
def test_p3_aol_spectral_bound(m, n, alpha):
    for seed in range(3):
        X = synth.power_law_matrix(m, n, alpha, seed)
        X1 = O.preconditioned(X, "aol")
        assert np.linalg.norm(X1, 2) <= 1 + 1e-14
        G = X @ X.T if m <= n else X.T @ X
        assert np.abs(G).sum(1).max() >= np.linalg.eigvalsh(G).max() * (1 - 1e-14)
    heavy = np.random.default_rng(4).standard_cauchy((40, 70))
    assert np.linalg.norm(O.preconditioned(heavy, "aol"), 2) <= 1 + 1e-14
    assert np.linalg.norm(O.preconditioned(X, "frobenius"), 2) <= 1 + 1e-14


# --------------------------------------------------------------------------
# P4: output singular values lie in phi([sigma_min, sigma_max])
# --------------------------------------------------------------------------
@pytest.mark.parametrize("m,n", [(64, 576), (256, 256), (300, 120)])
def test_p4_singular_value_band(m, n):
    X = synth.power_law_matrix(m, n, 1.0, seed=2)
    sv1 = np.linalg.svd(O.preconditioned(X, "aol"), compute_uv=False)
    grid = np.linspace(sv1.min(), sv1.max(), 200001)
    img = phi(grid, [TRIPLE] * 4)
    lo, hi = img.min(), img.max()
    svo = np.linalg.svd(O.orthogonalize(X, 4), compute_uv=False)
    assert svo.min() >= lo - 1e-9 and svo.max() <= hi + 1e-9
    # the constant triple's image never leaves (0, 1.2024] for inputs in [1e-2, 1]
    g = phi(np.linspace(1e-2, 1.0, 100001), [TRIPLE] * 4)
    assert g.min() > 0 and g.max() < 1.2024


# --------------------------------------------------------------------------
# P6: invariances
# --------------------------------------------------------------------------
def signed_perm(rng, n):
    P = np.zeros((n, n))
    P[np.arange(n), rng.permutation(n)] = rng.choice([-1.0, 1.0], n)
    return P


@pytest.mark.parametrize("m,n", [(20, 35), (35, 20), (24, 24)])
def test_p6_invariances(m, n):
    rng = np.random.default_rng(m * n)
    X = synth.power_law_matrix(m, n, 0.8, seed=4)
    Z = O.orthogonalize(X, 4)
    for alpha in (3.7, -0.02):
        assert relF(O.orthogonalize(alpha * X, 4), np.sign(alpha) * Z) <= 1e-12
        Zf = O.orthogonalize(X, 5, None, "frobenius")
        assert relF(O.orthogonalize(alpha * X, 5, None, "frobenius"), np.sign(alpha) * Zf) <= 1e-12
    X1f = O.preconditioned(X, "frobenius")
    assert abs(np.linalg.norm(X1f) - 1.0) <= 1e-14
    P, R = signed_perm(rng, m), signed_perm(rng, n)
    assert relF(O.orthogonalize(P @ X @ R, 4), P @ Z @ R) <= 1e-12
    U, V = rand_orth(rng, m), rand_orth(rng, n)
    Zf = O.orthogonalize(X, 5, None, "frobenius")
    assert relF(O.orthogonalize(U @ X @ V, 5, None, "frobenius"), U @ Zf @ V) <= 1e-11
    if m != n:
        assert relF(O.orthogonalize(X.T, 4), Z.T) <= 1e-13
    assert relF(O.orthogonalize(X, 4, side="cols"), O.orthogonalize(X.T, 4, side="rows").T) <= 1e-13


# --------------------------------------------------------------------------
# Block-diagonal inputs: every product of the iteration (eq. ns_quintic) keeps
# the block structure of X X^T, and the AOL scale of a row (Section 4.1)
# only sums that row of the Gram, so the output is the block-diagonal of the
# blocks' own outputs.  A global normalisation (Frobenius) couples the blocks.
# --------------------------------------------------------------------------
@pytest.mark.parametrize("m,n,count", [(40, 40, 4), (30, 52, 5), (61, 23, 3), (7, 9, 7)])
def test_block_diagonal_input_gives_block_diagonal_output(m, n, count):
    layout, blocks = synth.block_diagonal_blocks(m, n, count, 0.7, seed=11)
    X = np.zeros((m, n))
    for (r0, r1, c0, c1), B in zip(layout, blocks):
        X[r0:r1, c0:c1] = B
    for precond in ("aol", "none"):
        Z = O.orthogonalize(X, 4, None, precond)
        E = Z.copy()
        for (r0, r1, c0, c1), B in zip(layout, blocks):
            Zb = O.orthogonalize(B, 4, None, precond)
            assert relF(Z[r0:r1, c0:c1], Zb) <= 1e-12, precond
            E[r0:r1, c0:c1] = 0
        assert np.max(np.abs(E)) <= 1e-14 * np.max(np.abs(Z)), precond
    Zf = O.orthogonalize(X, 4, None, "frobenius")
    r0, r1, c0, c1 = layout[0]
    assert relF(Zf[r0:r1, c0:c1], O.orthogonalize(blocks[0], 4, None, "frobenius")) > 1e-3


def test_block_diagonal_layout_partitions_and_orients():
    for m, n, count in [(65536, 65536, 256), (65536, 40000, 128), (40000, 65536, 128), (5, 5, 5)]:
        lay = synth.block_diagonal_layout(m, n, count)
        assert len(lay) == count
        assert lay[0][0] == 0 and lay[0][2] == 0 and lay[-1][1] == m and lay[-1][3] == n
        for a, b in zip(lay, lay[1:]):
            assert a[1] == b[0] and a[3] == b[2]
        for r0, r1, c0, c1 in lay:
            assert (m <= n) == (r1 - r0 <= c1 - c0)
    with pytest.raises(ValueError):
        synth.block_diagonal_layout(5, 4, 4)          # a square 1 x 1 block in a tall matrix
    with pytest.raises(ValueError):
        synth.block_diagonal_layout(4, 4, 5)


# --------------------------------------------------------------------------
# P7: Lemma 1, <G, PolarFactor(G S)> > 0, and the same for the t = 4 output
# --------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(4))
def test_p7_descent_alignment(seed):
    rng = np.random.default_rng(seed)
    G = rng.standard_cauchy((30, 50))
    S = np.diag(rng.uniform(0.01, 10.0, 50))
    assert np.sum(G * O.polar_factor(G @ S)) > 0
    for X in (G, synth.power_law_matrix(64, 256, 1.0, seed)):
        assert np.sum(X * O.orthogonalize(X, 4)) > 0


# --------------------------------------------------------------------------
# Metrics of Section 3 and the bias appendix
# --------------------------------------------------------------------------
def test_metric_definitions():
    X = synth.power_law_matrix(30, 45, 0.8, seed=0)
    Q = O.polar_factor(X)
    assert O.eps_polar(np.zeros_like(X), X) == pytest.approx(1.0, abs=1e-14)
    assert O.eps_polar(Q, X) <= 1e-14 and O.eps_ortho(Q) <= 1e-13
    assert O.eps_ortho(np.zeros_like(X)) == pytest.approx(1.0, abs=1e-14)
    Z = O.orthogonalize(X, 4)
    assert O.eps_polar(Z, X) <= O.eps_bias(X) + O.eps_approx(Z, X) + 1e-14


def test_rel_frobenius_by_hand():
    """||Z - R||_F / ||R||_F on 2 x 2 cases computed by hand: the reference (second
    argument) sets the scale, a zero reference falls back to the absolute error."""
    Z = np.array([[1.0, 2.0], [3.0, 4.0]])
    R = np.array([[1.0, 2.0], [3.0, 5.0]])
    assert O.rel_frobenius(Z, R) == pytest.approx(1.0 / np.sqrt(39.0), rel=1e-15)
    assert O.rel_frobenius(R, Z) == pytest.approx(1.0 / np.sqrt(30.0), rel=1e-15)
    assert O.rel_frobenius(R, R) == 0.0
    assert O.rel_frobenius(-R, R) == pytest.approx(2.0, rel=1e-15)
    assert O.rel_frobenius(np.zeros((2, 2)), R) == pytest.approx(1.0, rel=1e-15)
    assert O.rel_frobenius(Z, np.zeros((2, 2))) == pytest.approx(np.sqrt(30.0), rel=1e-15)
    # 3 x 4 with a difference of known norm 5 (a 3-4-5 pair) against ||R||_F = 10
    R3 = np.zeros((3, 4))
    R3[0, 0], R3[2, 3] = 6.0, 8.0
    Z3 = R3.copy()
    Z3[1, 1] += 3.0
    Z3[1, 2] -= 4.0
    assert O.rel_frobenius(Z3, R3) == pytest.approx(0.5, rel=1e-15)


def test_eps_ortho_tall_and_wide_by_hand():
    """The orthogonality error is taken on the min(m, n) side and normalised by
    sqrt(min(m, n)): a tall matrix with orthonormal columns scores 0 (its m x m
    Gram O O^T is a rank-k projector, far from I_m), a zero matrix 1, twice an
    orthonormal set ||3 I_k||_F / sqrt(k) = 3, and transposing changes nothing."""
    rng = np.random.default_rng(4)
    Q = rand_orth(rng, 7)[:, :3]                  # 7 x 3, Q^T Q = I_3
    assert O.eps_ortho(Q) <= 1e-14
    assert O.eps_ortho(Q.T) <= 1e-14
    P = Q @ Q.T                                   # the other side: a projector of rank 3
    assert np.linalg.norm(P - np.eye(7)) / np.sqrt(7) == pytest.approx(np.sqrt(4 / 7), rel=1e-12)
    assert O.eps_ortho(np.zeros((7, 3))) == pytest.approx(1.0, rel=1e-15)
    assert O.eps_ortho(np.zeros((3, 7))) == pytest.approx(1.0, rel=1e-15)
    assert O.eps_ortho(2.0 * Q) == pytest.approx(3.0, rel=1e-13)
    E = np.array([[1.0, 0.0], [0.0, 2.0], [0.0, 0.0]])   # E^T E = diag(1, 4)
    assert O.eps_ortho(E) == pytest.approx(3.0 / np.sqrt(2.0), rel=1e-15)
    assert O.eps_ortho(E.T) == pytest.approx(3.0 / np.sqrt(2.0), rel=1e-15)


# SCHEDULE5: five quintics normalised at 1 (p(1) = 1, p'(1) = 0), decreasing a.

def test_schedule_last_keeps_the_last_rows():
    """Appendix on the tuning of Newton-Schulz coefficients: fewer iterations from a
    five-iteration schedule keep its last rows.  Running the whole schedule equals
    running its first row, then the truncated schedule of the remaining iterations
    on that result (no second pre-conditioning): the retained rows must be the
    last ones, in order."""
    for a, b, c in SCHEDULE5:
        assert a + b + c == pytest.approx(1.0, abs=1e-15)
        assert a + 3 * b + 5 * c == pytest.approx(0.0, abs=1e-14)
    assert O.schedule_last(SCHEDULE5, 5) == SCHEDULE5
    assert O.schedule_last(SCHEDULE5, 1) == [SCHEDULE5[4]]
    assert O.schedule_last(SCHEDULE5, 0) == []
    assert O.schedule_last(SCHEDULE5, 3) == SCHEDULE5[2:]
    with pytest.raises(ValueError):
        O.schedule_last(SCHEDULE5, 6)
    X = synth.power_law_matrix(24, 40, 0.8, seed=3)
    for n in (4, 2):
        full = O.orthogonalize(X, 5, SCHEDULE5, "aol")
        head = O.orthogonalize(X, 5 - n, SCHEDULE5[:5 - n], "aol")
        tail = O.orthogonalize(head, n, O.schedule_last(SCHEDULE5, n), "none")
        assert relF(tail, full) <= 1e-13, n
    # the truncated run is the composition of the last n scalar polynomials
    X1 = O.preconditioned(X, "aol")
    Z = O.orthogonalize(X, 4, O.schedule_last(SCHEDULE5, 4), "aol")
    assert relF(Z, spectral_closed_form(X1.T, SCHEDULE5[1:]).T) <= 1e-12


# --------------------------------------------------------------------------
# P9: Figure 1a ordering, AOL starts closer to the polar factor than Frobenius
# --------------------------------------------------------------------------
@pytest.mark.parametrize("n", [64, 256])
def test_p9_fig1a_initial_polar_error_ordering(n):
    for seed in range(3):
        X = synth.gaussian_matrix(n, n, seed)
        Q = O.polar_factor(X)
        e_aol = O.eps_polar(O.preconditioned(X, "aol"), X, Q)
        e_frob = O.eps_polar(O.preconditioned(X, "frobenius"), X, Q)
        assert e_aol < e_frob


# --------------------------------------------------------------------------
# P5: Table 1, Muon baseline polar error 0.25 at 4096 (printed value)
# --------------------------------------------------------------------------
@pytest.mark.slow
def test_p5_table1_muon_baseline_polar_error():
    with open(os.path.join(HERE, "golden", "table1_ablation.json")) as f:
        gold = json.load(f)
    n = gold["n"]
    X = synth.gaussian_matrix(n, n, seed=0)
    Z = O.orthogonalize(X, gold["iters"], None, gold["precond"])
    e = O.eps_polar(Z, X)
    assert abs(e - gold["polar_error"]) <= gold["tolerance"]


# --------------------------------------------------------------------------
# Schatten-4 pre-conditioning (appendix on other pre-conditioning strategies)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("m,n", [(20, 35), (35, 20), (24, 24), (1, 9)])
def test_schatten4_scale_is_the_svd_norm(m, n):
    """X1 = X / (sum sigma^4)^(1/4): the Gram route equals LAPACK's singular values."""
    X = synth.power_law_matrix(m, n, 0.8, seed=m + n)
    sv = np.linalg.svd(X, compute_uv=False)
    s4 = np.sum(sv ** 4) ** 0.25
    assert relF(O.preconditioned(X, "schatten4"), X / s4) <= 1e-13
    assert relF(O.preconditioned(X, "schatten4", side="cols"), X / s4) <= 1e-13


def test_schatten4_bounds_and_rank_one():
    """sigma_max <= ||X||_S4 <= ||X||_F; equality for rank one, where X1 = u v^T."""
    for seed in range(3):
        X = synth.power_law_matrix(40, 70, 0.5, seed)
        X1 = O.preconditioned(X, "schatten4")
        assert np.linalg.norm(X1, 2) <= 1 + 1e-14
        assert np.linalg.norm(X1) >= 1 - 1e-14            # ||X||_F >= ||X||_S4
    rng = np.random.default_rng(3)
    u, v = rng.standard_normal(7), rng.standard_normal(11)
    X = 2.5 * np.outer(u, v)
    uv = np.outer(u / np.linalg.norm(u), v / np.linalg.norm(v))
    assert np.max(np.abs(O.preconditioned(X, "schatten4") - uv)) <= 1e-14
    assert np.max(np.abs(O.orthogonalize(X, 4, None, "schatten4") - phi(1.0, [TRIPLE] * 4) * uv)) <= 1e-13


@pytest.mark.parametrize("m,n", [(20, 35), (24, 24)])
def test_schatten4_invariances(m, n):
    """A spectral scale: orthogonal equivariance O(U X V) = U O(X) V and O(aX) = sign(a) O(X)."""
    rng = np.random.default_rng(m + 7 * n)
    X = synth.power_law_matrix(m, n, 0.8, seed=5)
    Z = O.orthogonalize(X, 4, None, "schatten4")
    U, V = rand_orth(rng, m), rand_orth(rng, n)
    assert relF(O.orthogonalize(U @ X @ V, 4, None, "schatten4"), U @ Z @ V) <= 1e-11
    assert relF(O.orthogonalize(-0.3 * X, 4, None, "schatten4"), -Z) <= 1e-12


@pytest.mark.parametrize("n", [64, 256, 512])
def test_schatten4_initial_polar_error_ordering(n):
    """The appendix figure of initialisations: Schatten-4 improves on Frobenius and AOL
    is better still (N(0,1) inputs).  Schatten-4 below Frobenius is also a theorem:
    every sigma_i / ||X||_S4 lies between sigma_i / ||X||_F and 1."""
    for seed in range(2):
        X = synth.gaussian_matrix(n, n, seed)
        Q = O.polar_factor(X)
        e = {p: O.eps_polar(O.preconditioned(X, p), X, Q) for p in ("frobenius", "schatten4", "aol")}
        assert e["aol"] < e["schatten4"] < e["frobenius"]


# --------------------------------------------------------------------------
# Optimizer step around the orthogonalization (Muon's step, orthogonalization replaced)
# --------------------------------------------------------------------------
def test_round_bf16_matches_the_storage_rounding():
    """The oracle's bf16 rounding equals an independent route: float32 -> bfloat16
    through NumPy's round-half-even on the scaled mantissa, and exact values stay."""
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-20, 20, 20000),
                        [0.0, -0.0, 1.0, -2.5, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -9]])
    got = O.round_bf16(x)
    f = x.astype(np.float32).astype(np.float64)
    e = np.floor(np.log2(np.abs(np.where(f == 0, 1.0, f))))
    q = 2.0 ** (e - 7)                                   # bf16 ulp for a normal value
    want = np.where(f == 0, f, np.round(f / q) * q)      # np.round: half to even
    assert np.array_equal(got, want)
    assert O.round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0          # tie to even
    assert O.round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6


def test_muon_momentum_is_a_geometric_series():
    """Constant gradient G from M = 0: after k steps M_k = G (1 - mu^k) / (1 - mu)."""
    G = synth.power_law_matrix(12, 20, 0.8, seed=1)
    W, M = np.zeros_like(G), np.zeros_like(G)
    mu = 0.9
    for k in range(1, 6):
        W, M, _ = O.muon_step(W, G, M, lr=0.01, momentum=mu, nesterov=False)
        assert np.max(np.abs(M - G * (1 - mu ** k) / (1 - mu))) <= 1e-13


def test_muon_nesterov_two_steps_by_hand():
    """Nesterov from M = 0: U1 = (1 + mu) G1; M1 = G1; U2 = G2 + mu (mu G1 + G2)."""
    G1 = synth.power_law_matrix(10, 16, 1.0, seed=2)
    G2 = synth.power_law_matrix(10, 16, 1.0, seed=3)
    mu, lr = 0.95, 0.1
    W0 = np.zeros_like(G1)
    W1, M1, O1 = O.muon_step(W0, G1, np.zeros_like(G1), lr, mu, nesterov=True)
    assert np.allclose(O1, O.orthogonalize(O.round_bf16((1 + mu) * G1), 4), rtol=0, atol=1e-14)
    W2, M2, O2 = O.muon_step(W1, G2, M1, lr, mu, nesterov=True)
    assert np.max(np.abs(M2 - (mu * G1 + G2))) <= 1e-14
    assert np.allclose(O2, O.orthogonalize(O.round_bf16(G2 + mu * (mu * G1 + G2)), 4), rtol=0, atol=1e-14)
    assert np.max(np.abs(W2 - (-lr * O1 - lr * O2))) <= 1e-14          # 10 x 16: scale 1


def test_muon_weight_decay_and_shape_scale():
    W = synth.power_law_matrix(30, 10, 1.0, seed=4)                      # tall: scale sqrt(3)
    Z = np.zeros_like(W)
    Wn, Mn, On = O.muon_step(W, Z, Z, lr=0.5, momentum=0.9, weight_decay=0.1)
    assert np.all(On == 0) and np.all(Mn == 0)
    assert np.max(np.abs(Wn - 0.95 * W)) <= 1e-15
    G = synth.power_law_matrix(30, 10, 1.0, seed=5)
    W1, _, O1 = O.muon_step(Z, G, Z, lr=1.0, momentum=0.0, nesterov=False)
    assert np.max(np.abs(W1 + np.sqrt(3.0) * O1)) <= 1e-14
    W2, _, _ = O.muon_step(Z, G, Z, lr=1.0, momentum=0.0, nesterov=False, shape_scale=False)
    assert np.max(np.abs(W2 + O1)) <= 1e-14
    # decoupled decay shrinks the old weights only, not the new step
    W3, _, O3 = O.muon_step(W, G, Z, lr=0.5, momentum=0.0, nesterov=False, weight_decay=0.1)
    assert np.max(np.abs(W3 - (0.95 * W - 0.5 * np.sqrt(3.0) * O3))) <= 1e-14
    assert np.max(np.abs(W3 - 0.95 * (W - 0.5 * np.sqrt(3.0) * O3))) > 1e-3


@pytest.mark.parametrize("seed", range(3))
def test_muon_step_is_a_descent_direction(seed):
    """Without momentum the step -lr O satisfies <G, W - W'> > 0 (Lemma 1's alignment)."""
    G = np.random.default_rng(seed).standard_cauchy((24, 40))
    W = np.zeros_like(G)
    Wn, _, _ = O.muon_step(W, G, np.zeros_like(G), lr=0.1, momentum=0.0, nesterov=False)
    assert np.sum(G * (W - Wn)) > 0

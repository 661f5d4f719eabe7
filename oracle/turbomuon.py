"""Plain fp64 oracle of Turbo-Muon's orthogonalization (arXiv 2512.04632).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the HIP path.  Everything here is
float64 NumPy; matrix products use NumPy's BLAS, the polar factor uses
LAPACK's SVD.  No blocking, fusion or reordering beyond the paper's steps.

Notation follows the paper: X0 is the input, A_k = X_k^T X_k the Gram matrix,
B_k = b A_k + c A_k A_k the polynomial, X_{k+1} = a X_k + X_k B_k the update
(Algorithm 1, the "Newton-Schulz Muon/Muon+" box of Section 4), and
Algorithm 2 (the "Newton-Schulz Turbo-Muon" box) replaces the Frobenius
scaling of the first iteration by the AOL vector
s_i = 1 / sqrt(sum_j |A_0|_{ij}) of eq. (aol) (Section 4.1).

Readings where the paper is silent or ambiguous (each is repeated in the
design notes):
* Side of the Gram.  Algorithm 2 forms X0^T X0 and scales columns.  A wide
  input (m <= n, square included) is handled as Algorithm 2 applied to its
  transpose, so the Gram is the m x m matrix X X^T and AOL scales rows; a tall
  input (m > n) follows Algorithm 2 literally.  The Gram is therefore always
  min(m, n) square, matching the O(min(m, n)) memory remark of Section 4.1.
* A_1 = s^T A_0 s in Algorithm 2 is read as diag(s) A_0 diag(s), and
  X_1 = X_0 s as X_0 diag(s) (a broadcast over columns).
* A zero row sum gives s_i = 0 (no epsilon); a zero Frobenius norm gives a
  zero X_1.
* One "iteration" is one (Gram, polynomial, update) triple; the AOL Gram is the
  Gram of iteration 1, so t iterations form exactly t Gram matrices.
* Coefficients: a list of (a_k, b_k, c_k), one per iteration; the default is
  the constant triple (3.4445, -4.7750, 2.0315) for every iteration, since the
  paper prints no schedule.
"""
from __future__ import annotations

from typing import Iterable, Sequence

import numpy as np

CONSTANT_TRIPLE = (3.4445, -4.7750, 2.0315)

PRECONDS = ("none", "frobenius", "aol", "schatten4")


def _coeff_list(t: int, coeffs) -> list:
    if coeffs is None:
        return [CONSTANT_TRIPLE] * t
    cl = [tuple(float(v) for v in row) for row in coeffs]
    if len(cl) != t or any(len(r) != 3 for r in cl):
        raise ValueError("coeffs must hold one (a, b, c) triple per iteration")
    return cl


def aol_vector(A0: np.ndarray) -> np.ndarray:
    """AOL vector of Algorithm 2, second line / eq. (aol).

    s_i = 1 / sqrt(||A0_i||_1): the inverse square root of the L1 norm of row i
    of the Gram matrix.  A zero row sum maps to s_i = 0.
    """
    r = np.abs(A0).sum(axis=1)
    s = np.zeros_like(r)
    pos = r > 0
    s[pos] = 1.0 / np.sqrt(r[pos])
    return s


def aol(X0: np.ndarray) -> np.ndarray:
    """AOL(X0) = X0 diag(sum_j |X0^T X0|_ij)^(-1/2), eq. (aol): column scaling."""
    X0 = np.asarray(X0, dtype=np.float64)
    s = aol_vector(X0.T @ X0)
    return X0 * s[None, :]


def frobenius_scale(X0: np.ndarray) -> np.ndarray:
    """X1 = X0 / ||X0||_F, Algorithm 1 first two lines (zero stays zero)."""
    X0 = np.asarray(X0, dtype=np.float64)
    f = np.linalg.norm(X0)
    if f == 0:
        return np.zeros_like(X0)
    return X0 * (1.0 / f)


def schatten4_scale(A0: np.ndarray) -> float:
    """1 / ||X0||_S4 from the first Gram (appendix on other pre-conditionings).

    ||X||_S4 = (sum_i sigma_i^4)^(1/4), and the eigenvalues of A0 = X0^T X0 are
    the sigma_i^2, so ||X||_S4 = ||A0||_F^(1/2): the scale comes from the
    Frobenius norm of the Gram Algorithm 2 forms anyway.  A zero Gram maps to 0.
    """
    f = np.linalg.norm(A0)
    return 0.0 if f == 0 else 1.0 / np.sqrt(f)


def first_iterate(X0: np.ndarray, precond: str = "aol"):
    """The pre-conditioned starting point X1 and its Gram A1 = X1^T X1.

    "aol" (Algorithm 2, eq. (aol)): the Gram A0 of the raw input gives the
    column scales s; X1 = X0 diag(s), and A1 = diag(s) A0 diag(s) is obtained
    by rescaling A0 rather than by a second product.  "frobenius" (Algorithm 1):
    X1 = X0 / ||X0||_F with its own Gram.  "schatten4" (appendix on other
    pre-conditionings): the uniform scale g = 1 / ||X0||_S4 = ||A0||_F^(-1/2)
    from the same first Gram, X1 = g X0 and A1 = g^2 A0.  "none": X1 = X0.
    """
    if precond not in PRECONDS:
        raise ValueError(f"unknown precond {precond!r}")
    X0 = np.asarray(X0, dtype=np.float64)
    if precond == "frobenius":
        X1 = frobenius_scale(X0)
        return X1, X1.T @ X1
    if precond == "none":
        X1 = X0.copy()
        return X1, X1.T @ X1
    A0 = X0.T @ X0
    if precond == "aol":
        s = aol_vector(A0)
        return X0 * s[None, :], (s[:, None] * A0) * s[None, :]
    g = schatten4_scale(A0)
    return X0 * g, A0 * (g * g)


def quintic_step(X: np.ndarray, A: np.ndarray, a: float, b: float, c: float) -> np.ndarray:
    """eq. (ns_quintic): a X + b X (X^T X) + c X (X^T X)^2, written with the
    Gram A = X^T X as a X + X (b A + c A^2), so that the quintic costs one
    Gram, one square of it and one product with X."""
    return a * X + X @ (b * A + c * (A @ A))


def newton_schulz(X0: np.ndarray, t: int, coeffs=None, precond: str = "aol") -> np.ndarray:
    """t quintic Newton-Schulz steps on the pre-conditioned X1 (Algorithms 1 and 2).

    The Gram used by the first step is the A1 of first_iterate (for AOL and
    Schatten-4, a rescaling of the Gram that gave the scale); every later step
    forms the Gram of its own iterate.  Step k uses the k-th (a, b, c) of
    coeffs (default: the constant triple).  t = 0 returns X1.
    """
    if t < 0:
        raise ValueError("t must be >= 0")
    cl = _coeff_list(t, coeffs)
    X, A = first_iterate(X0, precond)
    for k, (a, b, c) in enumerate(cl):
        if k > 0:
            A = X.T @ X
        X = quintic_step(X, A, a, b, c)
    return X


def schedule_last(schedule, n: int) -> list:
    """Fewer iterations from a schedule designed for more (appendix on the
    tuning of Newton-Schulz coefficients): of a schedule of T rows (a_k, b_k,
    c_k), n <= T iterations keep its n last rows, in their order."""
    rows = [tuple(float(v) for v in r) for r in schedule]
    T = len(rows)
    if not 0 <= n <= T:
        raise ValueError(f"cannot run {n} iterations from a schedule of {T} rows")
    return [rows[T - n + i] for i in range(n)]


def orthogonalize(X: np.ndarray, t: int = 4, coeffs=None, precond: str = "aol",
                  side: str = "auto") -> np.ndarray:
    """Orthogonalize an m x n matrix with the Gram on its smaller side.

    side="auto": a wide or square input (m <= n) runs Algorithm 2 on X^T and is
    transposed back (Gram X X^T, AOL scales rows); a tall input runs it as
    printed (Gram X^T X, AOL scales columns).  side="cols" runs Algorithm 2 on
    X as printed whatever its shape; side="rows" always on X^T.
    """
    X = np.asarray(X, dtype=np.float64)
    if X.ndim != 2:
        raise ValueError("X must be 2-D")
    m, n = X.shape
    if side == "auto":
        side = "rows" if m <= n else "cols"
    if side == "rows":
        return newton_schulz(X.T, t, coeffs, precond).T
    if side == "cols":
        return newton_schulz(X, t, coeffs, precond)
    raise ValueError(f"unknown side {side!r}")


def preconditioned(X: np.ndarray, precond: str = "aol", side: str = "auto") -> np.ndarray:
    """X1 of Algorithm 1 / 2 in the orientation of orthogonalize (t = 0)."""
    return orthogonalize(X, 0, None, precond, side)


# ---------------------------------------------------------------------------
# Exact references and metrics (Section 3 definitions, appendix on the bias)
# ---------------------------------------------------------------------------

def polar_factor(X: np.ndarray) -> np.ndarray:
    """PolarFactor(X) = U V^T from the thin SVD X = U Sigma V^T (Section 3)."""
    U, _, Vt = np.linalg.svd(np.asarray(X, dtype=np.float64), full_matrices=False)
    return U @ Vt


def eps_ortho(O: np.ndarray) -> np.ndarray:
    """Normalised orthogonality error ||O O^T - I||_F / sqrt(k) on the small side.

    Section 3 defines ||X^T X - I||_F; for a non-square O the Gram is taken on
    the min(m, n) side (the only side that can be the identity) and divided by
    sqrt(min(m, n)) so that a zero matrix scores 1.
    """
    O = np.asarray(O, dtype=np.float64)
    G = O @ O.T if O.shape[0] <= O.shape[1] else O.T @ O
    k = G.shape[0]
    return np.linalg.norm(G - np.eye(k)) / np.sqrt(k)


def eps_polar(Z: np.ndarray, X: np.ndarray, Q: np.ndarray | None = None) -> float:
    """eps_polar(Z, X) = ||Z - PolarFactor(X)||_F / sqrt(min(m, n)) (Section 3)."""
    if Q is None:
        Q = polar_factor(X)
    k = min(Q.shape)
    return float(np.linalg.norm(np.asarray(Z, dtype=np.float64) - Q) / np.sqrt(k))


def eps_bias(X: np.ndarray, side: str = "auto") -> float:
    """||Q - Q_aol||_F / sqrt(k): polar factors of X and of AOL(X) (bias appendix)."""
    Xa = preconditioned(X, "aol", side)
    return eps_polar(polar_factor(Xa), X)


def eps_approx(Z: np.ndarray, X: np.ndarray, side: str = "auto") -> float:
    """||Q_aol - NS_t(AOL(X))||_F / sqrt(k) for Z = NS_t(AOL(X)) (bias appendix)."""
    Xa = preconditioned(X, "aol", side)
    return eps_polar(Z, Xa)


def rel_frobenius(Z: np.ndarray, R: np.ndarray) -> float:
    """||Z - R||_F / ||R||_F."""
    R = np.asarray(R, dtype=np.float64)
    d = np.linalg.norm(np.asarray(Z, dtype=np.float64) - R)
    r = np.linalg.norm(R)
    return float(d / r) if r > 0 else float(d)


# ---------------------------------------------------------------------------
# Optimizer step around the orthogonalization
# ---------------------------------------------------------------------------

def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest bfloat16 (ties to even), as float64.

    Written out on the bit pattern of the float32 value: keep the top 16 bits,
    adding half an ulp of the kept part plus its lowest bit (round half to even).
    """
    f = np.ascontiguousarray(x, dtype=np.float32)
    b = f.view(np.uint32).astype(np.uint64)
    b = ((b + 0x7FFF + ((b >> 16) & 1)) >> 16) << 16
    out = b.astype(np.uint32).view(np.float32).astype(np.float64)
    out[np.isnan(f)] = np.nan
    return out


def muon_step(W: np.ndarray, G: np.ndarray, M: np.ndarray, lr: float, momentum: float,
              nesterov: bool = True, weight_decay: float = 0.0, t: int = 4, coeffs=None,
              precond: str = "aol", shape_scale: bool = True):
    """One step of Muon with the orthogonalization replaced by this method.

    The paper uses Turbo-Muon as a drop-in replacement of Muon's
    orthogonalization and keeps the rest of Muon's step; that step is read as
    heavy-ball momentum on the gradient, optionally in Nesterov form, followed
    by the orthogonalized update (the steepest-descent appendix writes the
    update as -eta PolarFactor(G S)):

        M' = momentum M + G
        U  = G + momentum M'   (nesterov)   or   U = M'
        O  = orthogonalize(bf16(U), t, coeffs, precond)
        W' = W (1 - lr weight_decay) - lr scale O,
             scale = sqrt(max(1, rows / cols)) if shape_scale else 1.

    U is rounded to bfloat16 first because that is the storage the
    orthogonalization runs in.  Returns (W', M', O).
    """
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    M = np.asarray(M, dtype=np.float64)
    Mn = momentum * M + G
    U = G + momentum * Mn if nesterov else Mn
    O = orthogonalize(round_bf16(U), t, coeffs, precond)
    m, n = W.shape
    scale = np.sqrt(max(1.0, m / n)) if shape_scale else 1.0
    Wn = W * (1.0 - lr * weight_decay) - lr * scale * O
    return Wn, Mn, O

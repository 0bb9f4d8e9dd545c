"""Plain fp64 CPU oracle for ExTernD (Expanded-rank Ternary Decomposition).

TEST INFRASTRUCTURE ONLY -- see ``oracle/__init__.py``.  The product path
(the HIP library and its Python binding) never imports this module.

What it computes (paper: "ExTernD: Expanded-Rank Ternary Decomposition",
Sec. 2):

* ``ternarize``            -- the adaptive mean-threshold operator T_tau,
                              Eq. (2), Sec. 2.2, with its keep-largest rule.
* ``factorize_sequential`` -- greedy sequential ALS, Sec. 2.3 ("mode S"):
                              one component at a time, alternating ternary
                              fit, optimal scale, rank-one deflation.  With
                              importance weights it applies Sec. 2.5.
                              Optional single-entry safeguard of
                              Proposition 2 (Appendix A).
* ``factorize_block``      -- batched block ALS, Sec. 2.4 ("mode B"):
                              decorrelated least-squares targets, Eq. (3),
                              joint exact scale solve, Eq. (4), block
                              deflation; weighted variant of Sec. 2.5 with
                              the plain-residual V-step.
* step functions           -- ``init_block``, ``vstep``, ``ustep``,
                              ``scale_solve``, ``deflate``: one step each of
                              mode B, for per-step parity on injected state.
* ``optimal_projection``   -- closed-form optimal ternary projection
                              mentioned in Sec. 2.2 (test aid only).
* ``bruteforce_rank1``     -- exhaustive best ternary rank-one fit on tiny
                              matrices (test aid only).
* ``refine``, ``refine_block`` -- refinement sweeps of Sec. 2.4: each
                              block in turn is added back to the residual,
                              fitted again and deflated again.
* ``apply``                -- inference y = B (diag(D) (C x)), the cost
                              model of Sec. 2.6, written as its definition.

Everything is float64.  Library primitives (matmul, linear solve, stable
sort) serve as single steps; there is no blocking, fusion or reordering
beyond what the paper states.

Readings taken where the paper is silent (each also listed in the design doc):

* R1 (initialisation, silent in Sec. 2.3/2.4): the first partner vector is
  u = T_tau(R[:, j*]) for the residual column j* with the largest weighted
  energy h~_j * ||R[:, j]||^2; a block uses the top-bb such columns in
  descending order.  Ties go to the smaller column index.
* R2 (iteration): one ALS iteration is a V-step followed by a U-step, in the
  order printed in Sec. 2.3; the scale uses the final u and v.  The count is
  an argument (the paper uses 15).
* R3 (ridge in Eq. (3)): eps = 1e-6 * trace(G) / bb for each Gram matrix G.
  When trace(G) == 0 every column is zero and the target is zero.
* R4 (scale solve, Eq. (4)): (M + delta I) d = g with
  delta = 1e-12 * trace(M) / bb (a guard, not a regularizer: its relative
  effect on d is ~1e-12).  trace(M) == 0 gives d = 0.  Mode S uses the
  literal Sec. 2.3 formula with d = 0 when the denominator is 0.
* R5 (T_tau): strict ">" against tau * mean|x| over the vector's own
  length; the fallback keeps the largest |x_i| with the smallest index; an
  all-zero vector maps to zero.
* R6 (rank): k = floor(mu * min(m, n) + 0.5).
* R7 (block cap, Sec. 2.4): b_eff = min(block, max(1, floor(min(m,n)/8)));
  the last block holds k - c0 components.
* R8 (weights, Sec. 2.5): h~ = h / max(h) + lambda, one weight per column
  of A; lambda defaults to 0 (the setting the paper uses).  The U-step
  target is R diag(h~) V with Gram V^T diag(h~) V; the V-step uses the
  plain residual R and U^T U; the scale solve uses (U^T U) o (V^T diag(h~) V)
  and diag(U^T R diag(h~) V).
* R9 (energies): E = 1 - ||R||_F^2 / ||A||_F^2 (Sec. 2.1); the weighted
  energy is E_w = 1 - sum_j h~_j ||R_:j||^2 / sum_j h~_j ||A_:j||^2.  A zero
  matrix has E = 1.
* R10 (energy target, Sec. 1 and Sec. 3: mu chosen per matrix so that a
  target accuracy is met exactly): the run stops after the first block
  whose energy reaches the target (E, or E_w when weights are given, the
  objective that run minimizes), or at k = rank_of(m, n, mu_max).  Greedy
  deflation makes the result the prefix of the full mu_max run, so this is
  the smallest block-multiple k that meets the target.
* R11 (refinement sweeps, Sec. 2.4, which only says a block is added back,
  fitted again and deflated again, and that energy improves monotonically):
  blocks are revisited in extraction order.  The fit is warm-started from the
  block's current U and runs the same ``iters`` V-step/U-step iterations and
  joint scale solve as extraction.  The new block replaces the old one only
  when the energy it removes from R' = R + U diag(d) V^T,
  2 d'^T g' - d'^T M' d' (the weighted objective when weights are given),
  is strictly larger than what the old block removes, ||R'||^2 - ||R||^2;
  otherwise the old block stays.  Every revisit therefore leaves the
  objective no worse, which is the monotone improvement the paper states.
* R12 (safeguard for blocks; Proposition 2 augments each sequential step
  with the single residual entry of largest magnitude): after a block's
  ALS and Eq. (4) scales, the energy the block removes, 2 d^T g - d^T M d,
  is compared with max_ij R_ij^2; when the entry is strictly larger the
  block becomes that one component (u = e_i*, v = sign(R_i*j*) e_j*,
  d = |R_i*j*|, the first index in row-major order on ties) followed by
  bb - 1 zero components.  Every block then removes at least
  ||R||^2 / (m n), which gives Proposition 2's geometric bound per block;
  at bb = 1 it is the sequential augmented step.  Plain objective only.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

__all__ = [
    "RIDGE_REL", "SCALE_GUARD_REL",
    "rank_of", "effective_block", "normalized_weights",
    "ternarize", "ternarize_columns",
    "init_block", "vstep", "ustep", "scale_solve", "deflate",
    "energy", "Factorization",
    "factorize_sequential", "factorize_block", "apply",
    "refine_block", "refine", "Refinement",
    "optimal_projection", "bruteforce_rank1", "reconstruct",
]

RIDGE_REL = 1e-6          # reading R3
SCALE_GUARD_REL = 1e-12   # reading R4


# --------------------------------------------------------------------------
# sizes and weights
# --------------------------------------------------------------------------
def rank_of(m: int, n: int, mu: float) -> int:
    """Inner rank k = mu * min(m, n) (Sec. 2.1), rounded half up (R6)."""
    return int(math.floor(mu * min(m, n) + 0.5))


def effective_block(m: int, n: int, block: int) -> int:
    """Block width capped at floor(min(m, n) / 8) (Sec. 2.4; R7)."""
    return int(min(block, max(1, min(m, n) // 8)))


def normalized_weights(h: Optional[np.ndarray], n: int, lam: float = 0.0) -> np.ndarray:
    """h~ = h / max(h) + lambda (Sec. 2.5); ones if no h (lambda unused)."""
    if h is None:
        return np.ones(n, dtype=np.float64)
    h = np.asarray(h, dtype=np.float64)
    if h.shape != (n,) or not np.all(np.isfinite(h)) or np.any(h < 0) or h.max() <= 0:
        raise ValueError("importance weights must be finite, non-negative, not all zero")
    if not (math.isfinite(lam) and lam >= 0.0):
        raise ValueError("lambda must be finite and non-negative")
    return h / h.max() + lam


# --------------------------------------------------------------------------
# T_tau, Eq. (2)
# --------------------------------------------------------------------------
def ternarize(x: np.ndarray, tau: float) -> np.ndarray:
    """T_tau(x)_i = sign(x_i) * 1[|x_i| > tau * mean_j |x_j|]  (Eq. (2)).

    If no entry passes, the single largest |x_i| (smallest index on ties)
    keeps its sign (Sec. 2.2).  A zero vector maps to zero (R5).
    """
    x = np.asarray(x, dtype=np.float64)
    L = x.shape[0]
    a = np.abs(x)
    theta = tau * (np.sum(a) / L)
    t = np.where(a > theta, np.sign(x), 0.0)
    if not np.any(t):
        i = int(np.argmax(a))          # first index of the maximum
        t[i] = np.sign(x[i])           # stays 0 when x == 0
    return t.astype(np.int8)


def ternarize_columns(X: np.ndarray, tau: float) -> np.ndarray:
    """Apply T_tau to every column of X independently."""
    X = np.asarray(X, dtype=np.float64)
    out = np.empty(X.shape, dtype=np.int8)
    for c in range(X.shape[1]):
        out[:, c] = ternarize(X[:, c], tau)
    return out


# --------------------------------------------------------------------------
# one step each of the block ALS (Sec. 2.4, 2.5)
# --------------------------------------------------------------------------
def _ridge_solve(G: np.ndarray, rhs: np.ndarray) -> np.ndarray:
    """(G + eps I)^{-1} rhs with eps = RIDGE_REL * trace(G) / bb (R3)."""
    bb = G.shape[0]
    tr = float(np.trace(G))
    if tr == 0.0:
        return np.zeros(rhs.shape, dtype=np.float64)
    eps = RIDGE_REL * tr / bb
    return np.linalg.solve(G + eps * np.eye(bb), rhs)


def init_block(R: np.ndarray, w: np.ndarray, bb: int, tau: float):
    """Initial U for a block (reading R1).

    Columns are ranked by h~_j * ||R[:, j]||^2, descending, ties to the
    smaller index; U[:, c] = T_tau(R[:, J[c]]).  Returns (U, J).
    """
    s = w * np.sum(R * R, axis=0)
    order = np.argsort(-s, kind="stable")
    J = order[:bb]
    U = ternarize_columns(R[:, J], tau)
    return U, J


def vstep(R: np.ndarray, U: np.ndarray, tau: float):
    """V <- T_tau([(U^T U + eps I)^{-1} U^T R]^T), Eq. (3), first half.

    The V-target uses the plain residual also when weights are in use
    (Sec. 2.5).  Returns (V, Y) with V n x bb int8 and Y the bb x n target.
    """
    Uf = U.astype(np.float64)
    P = Uf.T @ R
    G = Uf.T @ Uf
    Y = _ridge_solve(G, P)
    V = ternarize_columns(Y.T, tau)
    return V, Y


def ustep(R: np.ndarray, V: np.ndarray, w: np.ndarray, tau: float):
    """U <- T_tau(W V (V^T H V + eps I)^{-1}), Eq. (3) second half, W = R diag(h~).

    Unweighted: h~ = 1 and this is U <- T_tau(R V (V^T V + eps I)^{-1}).
    Returns (U, Q, Z) with Q = R diag(h~) V and Z the m x bb target.
    """
    Vf = V.astype(np.float64)
    HV = w[:, None] * Vf
    Q = R @ HV
    G = Vf.T @ HV
    Z = _ridge_solve(G, Q.T).T       # G symmetric: Q G^{-1} = (G^{-1} Q^T)^T
    U = ternarize_columns(Z, tau)
    return U, Q, Z


def scale_solve(U: np.ndarray, V: np.ndarray, Q: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Joint scales from [(U^T U) o (V^T H V)] d = diag(U^T R H V), Eq. (4).

    Q = R H V from the last U-step (V has not changed since), so
    diag(U^T R H V) = column sums of U o Q.  Guarded solve per reading R4.
    """
    Uf = U.astype(np.float64)
    Vf = V.astype(np.float64)
    M = (Uf.T @ Uf) * (Vf.T @ (w[:, None] * Vf))
    g = np.sum(Uf * Q, axis=0)
    bb = M.shape[0]
    tr = float(np.trace(M))
    if tr == 0.0:
        return np.zeros(bb, dtype=np.float64)
    delta = SCALE_GUARD_REL * tr / bb
    return np.linalg.solve(M + delta * np.eye(bb), g)


def deflate(R: np.ndarray, U: np.ndarray, V: np.ndarray, d: np.ndarray) -> np.ndarray:
    """R <- R - U diag(d) V^T  (Sec. 2.4; rank-one form in Sec. 2.3)."""
    return R - (U.astype(np.float64) * d[None, :]) @ V.astype(np.float64).T


def energy(R: np.ndarray, A_fro2: float, w: Optional[np.ndarray] = None, A_col2: Optional[np.ndarray] = None):
    """E = 1 - ||R||^2/||A||^2 (Sec. 2.1) and, with weights, E_w (R9)."""
    col2 = np.sum(R * R, axis=0)
    E = 1.0 if A_fro2 == 0.0 else 1.0 - float(np.sum(col2)) / A_fro2
    if w is None:
        return E, None
    den = float(np.dot(w, A_col2))
    Ew = 1.0 if den == 0.0 else 1.0 - float(np.dot(w, col2)) / den
    return E, Ew


# --------------------------------------------------------------------------
# full factorizations
# --------------------------------------------------------------------------
@dataclass
class Factorization:
    B: np.ndarray                 # m x k int8 in {-1,0,1}
    C: np.ndarray                 # k x n int8 in {-1,0,1}
    D: np.ndarray                 # k float64
    E: float                      # plain energy preserved
    E_w: Optional[float]          # weighted energy (None without weights)
    curve: np.ndarray             # E after each component (S) or block (B)
    curve_w: Optional[np.ndarray]
    k: int
    block: int
    safeguard_fired: int = 0      # Prop. 2 single-entry step taken (S)
    safeguard_would_fire: int = 0 # single entry would beat ALS (S)
    fro2_curve: np.ndarray = field(default_factory=lambda: np.zeros(0))
    k_used: int = -1              # components extracted (R10 stop), else k


def factorize_sequential(A: np.ndarray, mu: float, tau: float, iters: int,
                         h: Optional[np.ndarray] = None, safeguard: bool = False,
                         k: Optional[int] = None, lam: float = 0.0) -> Factorization:
    """Greedy sequential ALS, Sec. 2.3 (mode S), weighted per Sec. 2.5.

    R <- A; for each component: u from reading R1, then ``iters`` times
    v <- T_tau(R^T u), u <- T_tau(R diag(h~) v); scale
    d = u^T R H v / (||u||^2 v^T H v) (Sec. 2.3, weighted Sec. 2.5);
    R <- R - d u v^T.  With ``safeguard`` the step of Proposition 2 is
    used: the single residual entry of largest magnitude replaces the ALS
    pair when it removes more energy (unweighted objective only).
    """
    A = np.asarray(A, dtype=np.float64)
    m, n = A.shape
    if k is None:
        k = rank_of(m, n, mu)
    w = normalized_weights(h, n, lam)
    weighted = h is not None
    if safeguard and weighted:
        raise ValueError("the safeguard of Proposition 2 is stated for the unweighted objective")
    R = A.copy()
    A_col2 = np.sum(A * A, axis=0)
    A_fro2 = float(np.sum(A_col2))
    B = np.zeros((m, k), dtype=np.int8)
    C = np.zeros((k, n), dtype=np.int8)
    D = np.zeros(k, dtype=np.float64)
    curve = np.zeros(k)
    curve_w = np.zeros(k) if weighted else None
    fro2 = np.zeros(k)
    fired = would = 0
    for i in range(k):
        s = w * np.sum(R * R, axis=0)
        j0 = int(np.argmax(s))
        u = ternarize(R[:, j0], tau).astype(np.float64)
        v = np.zeros(n)
        for _ in range(iters):
            v = ternarize(R.T @ u, tau).astype(np.float64)
            u = ternarize(R @ (w * v), tau).astype(np.float64)
        g = float(u @ R @ (w * v))
        den = float(u @ u) * float(v @ (w * v))
        d = g / den if den > 0 else 0.0
        if safeguard:
            gain_als = g * g / den if den > 0 else 0.0
            ii, jj = np.unravel_index(int(np.argmax(np.abs(R))), R.shape)
            gain_one = float(R[ii, jj]) ** 2
            if gain_one > gain_als:
                would += 1
                fired += 1
                u = np.zeros(m); u[ii] = 1.0
                v = np.zeros(n); v[jj] = 1.0 if R[ii, jj] >= 0 else -1.0
                d = abs(float(R[ii, jj]))
        elif not weighted:
            ii, jj = np.unravel_index(int(np.argmax(np.abs(R))), R.shape)
            if den > 0 and float(R[ii, jj]) ** 2 > g * g / den:
                would += 1
        R -= d * np.outer(u, v)
        B[:, i] = u.astype(np.int8)
        C[i, :] = v.astype(np.int8)
        D[i] = d
        E, Ew = energy(R, A_fro2, w if weighted else None, A_col2)
        curve[i] = E
        fro2[i] = float(np.sum(R * R))
        if weighted:
            curve_w[i] = Ew
    E, Ew = energy(R, A_fro2, w if weighted else None, A_col2)
    return Factorization(B, C, D, E, Ew, curve, curve_w, k, 1, fired, would, fro2)


def factorize_block(A: np.ndarray, mu: float, tau: float, block: int, iters: int,
                    h: Optional[np.ndarray] = None, k: Optional[int] = None,
                    max_blocks: Optional[int] = None, target: Optional[float] = None,
                    lam: float = 0.0, safeguard: bool = False) -> Factorization:
    """Batched block ALS with decorrelated targets, Sec. 2.4 (mode B).

    For each block of bb = min(b_eff, k - c0) components: U from reading R1,
    then ``iters`` times the V-step and U-step of Eq. (3); joint scales
    from Eq. (4); R <- R - U diag(d) V^T.  Deflation across blocks is
    sequential.  Weighted per Sec. 2.5 (reading R8).  ``max_blocks`` stops
    early (used only to time a bounded sample).  ``target``: stop after the
    first block whose energy reaches it (reading R10); the components past
    ``k_used`` stay zero and ``curve`` holds the blocks done.  ``safeguard``:
    the block analog of Proposition 2's augmented step (reading R12; plain
    objective only); ``safeguard_fired`` counts the blocks it replaced.
    """
    A = np.asarray(A, dtype=np.float64)
    m, n = A.shape
    if k is None:
        k = rank_of(m, n, mu)
    b_eff = effective_block(m, n, block)
    w = normalized_weights(h, n, lam)
    weighted = h is not None
    if safeguard and weighted:
        raise ValueError("the safeguard of Proposition 2 is stated for the unweighted objective")
    R = A.copy()
    A_col2 = np.sum(A * A, axis=0)
    A_fro2 = float(np.sum(A_col2))
    nblk = (k + b_eff - 1) // b_eff
    if max_blocks is not None:
        nblk = min(nblk, max_blocks)
    B = np.zeros((m, k), dtype=np.int8)
    C = np.zeros((k, n), dtype=np.int8)
    D = np.zeros(k, dtype=np.float64)
    curve = np.zeros(nblk)
    curve_w = np.zeros(nblk) if weighted else None
    fro2 = np.zeros(nblk)
    fired = 0
    for blk in range(nblk):
        c0 = blk * b_eff
        bb = min(b_eff, k - c0)
        U, _ = init_block(R, w, bb, tau)
        V = np.zeros((n, bb), dtype=np.int8)
        Q = np.zeros((m, bb))
        for _ in range(iters):
            V, _ = vstep(R, U, tau)
            U, Q, _ = ustep(R, V, w, tau)
        d = scale_solve(U, V, Q, w)
        if safeguard:
            # energy the block removes, 2 d^T g - d^T M d (Eq. (4)), against
            # the largest residual entry squared (Proposition 2, option (b))
            Uf, Vf = U.astype(np.float64), V.astype(np.float64)
            M = (Uf.T @ Uf) * (Vf.T @ Vf)
            g = np.sum(Uf * Q, axis=0)
            gain_blk = float(2.0 * (d @ g) - d @ M @ d)
            flat = int(np.argmax(np.abs(R)))   # first (row-major) index of the maximum
            ii, jj = divmod(flat, n)
            if float(R[ii, jj]) ** 2 > gain_blk:
                fired += 1
                U = np.zeros((m, bb), dtype=np.int8)
                V = np.zeros((n, bb), dtype=np.int8)
                d = np.zeros(bb)
                U[ii, 0] = 1
                V[jj, 0] = 1 if R[ii, jj] >= 0 else -1
                d[0] = abs(float(R[ii, jj]))
        R = deflate(R, U, V, d)
        B[:, c0:c0 + bb] = U
        C[c0:c0 + bb, :] = V.T
        D[c0:c0 + bb] = d
        E, Ew = energy(R, A_fro2, w if weighted else None, A_col2)
        curve[blk] = E
        fro2[blk] = float(np.sum(R * R))
        if weighted:
            curve_w[blk] = Ew
        if target is not None and (Ew if weighted else E) >= target:
            nblk = blk + 1
            curve, fro2 = curve[:nblk], fro2[:nblk]
            if weighted:
                curve_w = curve_w[:nblk]
            break
    E, Ew = energy(R, A_fro2, w if weighted else None, A_col2)
    k_used = min(nblk * b_eff, k)
    return Factorization(B, C, D, E, Ew, curve, curve_w, k, b_eff, fired, 0, fro2, k_used)


def _weighted_fro2(R: np.ndarray, w: np.ndarray) -> float:
    """sum_j h~_j ||R[:, j]||^2 (w = ones gives ||R||_F^2)."""
    return float(np.dot(w, np.sum(R * R, axis=0)))


def refine_block(R: np.ndarray, U: np.ndarray, V: np.ndarray, d: np.ndarray, w: np.ndarray,
                 tau: float, iters: int):
    """One revisit of a refinement sweep (Sec. 2.4; reading R11).

    R is the residual with the block (U m x bb, V n x bb, scales d) already
    deflated.  R' = R + U diag(d) V^T; the block ALS of Eq. (3) runs
    ``iters`` times from the current U; scales from Eq. (4).  The new block
    is kept when it removes strictly more of the objective from R' than the
    old one.  Returns (R_new, U, V, d, accepted, old_gain, new_gain).
    """
    Rp = R + (U.astype(np.float64) * d[None, :]) @ V.astype(np.float64).T
    old_gain = _weighted_fro2(Rp, w) - _weighted_fro2(R, w)
    Un = U
    Vn = V
    Q = np.zeros((R.shape[0], U.shape[1]))
    for _ in range(iters):
        Vn, _ = vstep(Rp, Un, tau)
        Un, Q, _ = ustep(Rp, Vn, w, tau)
    dn = scale_solve(Un, Vn, Q, w)
    # energy the new block removes from R': 2 d^T g - d^T M d, with
    # g = diag(U^T R' H V) and M = (U^T U) o (V^T H V) as in Eq. (4)
    Uf = Un.astype(np.float64)
    Vf = Vn.astype(np.float64)
    M = (Uf.T @ Uf) * (Vf.T @ (w[:, None] * Vf))
    g = np.sum(Uf * Q, axis=0)
    new_gain = float(2.0 * (dn @ g) - dn @ M @ dn)
    if new_gain > old_gain:
        return deflate(Rp, Un, Vn, dn), Un, Vn, dn, True, old_gain, new_gain
    return R, U, V, d, False, old_gain, new_gain


@dataclass
class Refinement:
    B: np.ndarray
    C: np.ndarray
    D: np.ndarray
    E: float
    E_w: Optional[float]
    sweep_curve: np.ndarray            # E after each sweep
    sweep_curve_w: Optional[np.ndarray]
    accepted: int                      # revisits that replaced their block
    revisits: int


def refine(A: np.ndarray, F: Factorization, tau: float, iters: int, sweeps: int,
           h: Optional[np.ndarray] = None, lam: float = 0.0) -> Refinement:
    """Refinement sweeps after a block factorization F of A (Sec. 2.4; R11).

    Each sweep revisits the blocks of F (width F.block, the last one
    partial) in order with ``refine_block``; R starts as A - B diag(D) C.
    """
    A = np.asarray(A, dtype=np.float64)
    m, n = A.shape
    w = normalized_weights(h, n, lam)
    weighted = h is not None
    B = F.B.copy()
    C = F.C.copy()
    D = np.asarray(F.D, dtype=np.float64).copy()
    k, b = F.k, F.block
    A_col2 = np.sum(A * A, axis=0)
    A_fro2 = float(np.sum(A_col2))
    R = A - reconstruct(B, D, C)
    nblk = (k + b - 1) // b
    curve = np.zeros(sweeps)
    curve_w = np.zeros(sweeps) if weighted else None
    accepted = 0
    for sw in range(sweeps):
        for blk in range(nblk):
            c0 = blk * b
            bb = min(b, k - c0)
            R, U, V, d, acc, _, _ = refine_block(R, B[:, c0:c0 + bb], C[c0:c0 + bb, :].T, D[c0:c0 + bb], w,
                                                 tau, iters)
            if acc:
                accepted += 1
                B[:, c0:c0 + bb] = U
                C[c0:c0 + bb, :] = V.T
                D[c0:c0 + bb] = d
        E, Ew = energy(R, A_fro2, w if weighted else None, A_col2)
        curve[sw] = E
        if weighted:
            curve_w[sw] = Ew
    if sweeps:
        E, Ew = curve[-1], (curve_w[-1] if weighted else None)
    else:
        E, Ew = energy(R, A_fro2, w if weighted else None, A_col2)
    return Refinement(B, C, D, E, Ew, curve, curve_w, accepted, sweeps * nblk)


def apply(B: np.ndarray, C: np.ndarray, D: np.ndarray, X: np.ndarray) -> np.ndarray:
    """Inference with a factorization, Sec. 2.6: y = B (diag(D) (C x)) for
    each row x of X (nb x n); returns Y (nb x m).  fp64."""
    T = np.asarray(C, dtype=np.float64) @ np.asarray(X, dtype=np.float64).T      # k x nb
    T = np.asarray(D, dtype=np.float64)[:, None] * T
    return (np.asarray(B, dtype=np.float64) @ T).T


def reconstruct(B: np.ndarray, D: np.ndarray, C: np.ndarray) -> np.ndarray:
    """A_hat = B diag(D) C, Eq. (1)."""
    return (B.astype(np.float64) * np.asarray(D, dtype=np.float64)[None, :]) @ C.astype(np.float64)


# --------------------------------------------------------------------------
# test aids
# --------------------------------------------------------------------------
def optimal_projection(u: np.ndarray):
    """Closed-form argmin_{t ternary, alpha} ||u - alpha t|| (Sec. 2.2).

    Sort |u| descending and keep the prefix of length s maximizing
    (1/sqrt(s)) * sum_{i<=s} |u|_(i); t takes the signs of u on that prefix.
    Returns (t, objective) with objective = (t^T u)^2 / ||t||^2.
    """
    u = np.asarray(u, dtype=np.float64)
    order = np.argsort(-np.abs(u), kind="stable")
    csum = np.cumsum(np.abs(u)[order])
    s_vals = np.arange(1, u.shape[0] + 1)
    score = csum / np.sqrt(s_vals)
    s_best = int(np.argmax(score)) + 1
    t = np.zeros(u.shape[0], dtype=np.int8)
    t[order[:s_best]] = np.sign(u[order[:s_best]]).astype(np.int8)
    obj = float(score[s_best - 1] ** 2)
    return t, obj


def bruteforce_rank1(R: np.ndarray):
    """Exhaustive max over ternary (u, v) != 0 of (u^T R v)^2 / (||u||^2 ||v||^2).

    By Proposition 1 this is the largest energy one ternary rank-one
    component can remove.  Only for tiny matrices (3^m * 3^n pairs).
    """
    R = np.asarray(R, dtype=np.float64)
    m, n = R.shape

    def all_ternary(L):
        grids = np.array(np.meshgrid(*([[-1, 0, 1]] * L), indexing="ij")).reshape(L, -1).T
        return grids[np.any(grids != 0, axis=1)].astype(np.float64)

    Us = all_ternary(m)
    Vs = all_ternary(n)
    G = Us @ R @ Vs.T
    den = np.sum(Us * Us, axis=1)[:, None] * np.sum(Vs * Vs, axis=1)[None, :]
    obj = G * G / den
    idx = np.unravel_index(int(np.argmax(obj)), obj.shape)
    return float(obj[idx]), Us[idx[0]].astype(np.int8), Vs[idx[1]].astype(np.int8)

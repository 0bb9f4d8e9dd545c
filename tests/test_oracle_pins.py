"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these compare the oracle with itself: each checks a worked value,
a closed form, a proposition of the paper, a brute-force enumeration, an
independent library route (least squares by SVD) or an exact symmetry.
"""
import math

import numpy as np
import pytest

import oracle
from paper_2607_13511_amd import synth


# --------------------------------------------------------------------------
# T_tau, Eq. (2): hand-worked values and invariants
# --------------------------------------------------------------------------
def test_ternarize_worked_values():
    # theta = 0.7 * (3 + 1 + 0.5 + 0) / 4 = 0.7875
    assert oracle.ternarize(np.array([3.0, -1.0, 0.5, 0.0]), 0.7).tolist() == [1, -1, 0, 0]
    # theta = 1.0 * 1 = 1: nothing is strictly above, the first largest entry is kept
    assert oracle.ternarize(np.array([1.0, 1.0, 1.0, 1.0]), 1.0).tolist() == [1, 0, 0, 0]
    # theta = 0.7: every entry passes
    assert oracle.ternarize(np.array([1.0, 1.0, 1.0, 1.0]), 0.7).tolist() == [1, 1, 1, 1]
    # fallback keeps the sign of the largest magnitude entry
    assert oracle.ternarize(np.array([0.2, -5.0, 0.1]), 3.0).tolist() == [0, -1, 0]
    # theta = 2 * (1+2+3+4)/4 = 5 : nothing passes, |4| at index 3 is kept
    assert oracle.ternarize(np.array([1.0, -2.0, 3.0, 4.0]), 2.0).tolist() == [0, 0, 0, 1]
    # the zero vector maps to zero
    assert oracle.ternarize(np.zeros(5), 0.7).tolist() == [0] * 5
    # strict inequality: an entry equal to the threshold is dropped
    # x = [2, 1, 0, 1]: mean|x| = 1, tau = 1 -> theta = 1; only 2 passes
    assert oracle.ternarize(np.array([2.0, 1.0, 0.0, -1.0]), 1.0).tolist() == [1, 0, 0, 0]


def test_ternarize_invariances():
    rng = np.random.default_rng(11)
    for _ in range(50):
        x = rng.standard_normal(rng.integers(1, 200))
        tau = float(rng.uniform(0.3, 2.5))
        t = oracle.ternarize(x, tau)
        assert np.array_equal(oracle.ternarize(8.0 * x, tau), t)       # positive power-of-two scale
        assert np.array_equal(oracle.ternarize(-x, tau), -t)            # odd
        assert np.count_nonzero(t) >= 1


@pytest.mark.parametrize("tau", [0.7, 1.0, 2.0])
def test_zero_fraction_closed_form(tau):
    # For Gaussian targets E|x| = sigma sqrt(2/pi), so
    # P(|x| <= tau E|x|) = erf(tau / sqrt(pi)): 42.35% / 57.51% / 88.95%.
    x = np.random.default_rng(123).standard_normal(1_000_000)
    zf = 1.0 - np.count_nonzero(oracle.ternarize(x, tau)) / x.size
    assert abs(zf - math.erf(tau / math.sqrt(math.pi))) < 3e-3


def test_factor_zero_fraction_matches_paper():
    # The paper states ~41% / ~57% / ~87% zeros at tau = 0.7 / 1.0 / 2.0
    # (Sec. 1, Sec. 3.2), almost independently of the matrix.
    A = synth.small("t4", 256, 512, 7)
    paper = {0.7: 0.41, 1.0: 0.57, 2.0: 0.87}
    prev = -1.0
    for tau, zf_paper in paper.items():
        f = oracle.factorize_block(A, 1.0, tau, 32, 8)
        zf = 0.5 * (np.mean(f.B == 0) + np.mean(f.C == 0))
        assert abs(zf - zf_paper) < 0.04, (tau, zf)
        assert zf > prev
        prev = zf


# --------------------------------------------------------------------------
# Proposition 1: exact per-step decrease; monotone energy
# --------------------------------------------------------------------------
@pytest.mark.parametrize("kind,m,n", [("gauss", 24, 17), ("t4_outliers", 40, 64), ("t4", 9, 33)])
def test_prop1_decrease_identity(kind, m, n):
    A = synth.small(kind, m, n, 5).astype(np.float64)
    f = oracle.factorize_sequential(A, 1.5, 0.7, 6)
    fro2 = np.concatenate([[np.sum(A * A)], f.fro2_curve])
    u2 = np.sum(f.B.astype(float) ** 2, axis=0)
    v2 = np.sum(f.C.astype(float) ** 2, axis=1)
    predicted = f.D ** 2 * u2 * v2          # = (u^T R v)^2 / (|u|^2 |v|^2) at the optimal d
    actual = fro2[:-1] - fro2[1:]
    assert np.all(actual >= -1e-14 * fro2[0])
    np.testing.assert_allclose(actual, predicted, rtol=1e-9, atol=1e-13 * fro2[0])


@pytest.mark.parametrize("weighted", [False, True])
def test_energy_monotone(weighted):
    A = synth.small("t4_rowscale", 96, 80, 3)
    h = synth.small_importance(80, 3) if weighted else None
    fs = oracle.factorize_sequential(A, 1.0, 1.0, 5, h=h)
    fb = oracle.factorize_block(A, 2.0, 1.0, 8, 5, h=h)
    for f in (fs, fb):
        c = f.curve_w if weighted else f.curve
        assert np.all(np.diff(c) >= -1e-12)
        assert c[0] > 0


# --------------------------------------------------------------------------
# brute force and the closed-form projection (Sec. 2.2)
# --------------------------------------------------------------------------
def test_rank1_step_against_bruteforce():
    rng = np.random.default_rng(5)
    hits = 0
    for _ in range(200):
        m, n = int(rng.integers(2, 5)), int(rng.integers(2, 5))
        R = rng.standard_normal((m, n))
        opt, _, _ = oracle.bruteforce_rank1(R)
        f = oracle.factorize_sequential(R, 1.0, 0.7, 8, k=1)
        dec = float(np.sum(R * R) - f.fro2_curve[0])
        assert -1e-12 <= dec <= opt * (1 + 1e-12) + 1e-15
        hits += abs(dec - opt) <= 1e-12 * opt
    # ALS is a heuristic; it still reaches the global optimum often on tiny cases
    assert hits >= 80


def test_optimal_projection_closed_form():
    rng = np.random.default_rng(9)
    for L in range(1, 11):
        for _ in range(5):
            u = rng.standard_normal(L)
            _, obj = oracle.optimal_projection(u)
            ts = np.array(np.meshgrid(*([[-1, 0, 1]] * L), indexing="ij")).reshape(L, -1).T
            ts = ts[np.any(ts != 0, axis=1)].astype(float)
            brute = np.max((ts @ u) ** 2 / np.sum(ts * ts, axis=1))
            assert abs(obj - brute) <= 1e-12 * brute


# --------------------------------------------------------------------------
# exact recovery of a ternary rank-one matrix
# --------------------------------------------------------------------------
@pytest.mark.parametrize("block", [1, 4])
def test_exact_rank1_recovery(block):
    rng = np.random.default_rng(21)
    m, n, alpha = 24, 40, 0.37
    u = rng.choice([-1, 0, 1], size=m, p=[0.3, 0.4, 0.3]); u[0] = 1
    v = rng.choice([-1, 0, 1], size=n, p=[0.3, 0.4, 0.3]); v[0] = -1
    A = alpha * np.outer(u, v)
    if block == 1:
        f = oracle.factorize_sequential(A, 1 / 24, 0.7, 4, k=1)
    else:
        f = oracle.factorize_block(A, 1 / 24, 0.7, block, 4, k=1)
    b, c, d = f.B[:, 0], f.C[0, :], f.D[0]
    sgn = 1 if np.array_equal(b, u) else -1
    assert np.array_equal(b, sgn * u) and np.array_equal(c, sgn * v)
    # mode B carries the 1e-12 relative guard of the scale solve
    assert abs(d - alpha) < (1e-15 if block == 1 else 1e-11 * alpha)
    assert f.E > 1 - 1e-14


# --------------------------------------------------------------------------
# Eq. (3) and Eq. (4) against independent least-squares routes
# --------------------------------------------------------------------------
def test_decorrelated_targets_are_least_squares():
    A = synth.small("t4", 120, 90, 8).astype(np.float64)
    w = oracle.normalized_weights(synth.small_importance(90, 8), 90)
    U, _ = oracle.init_block(A, np.ones(90), 6, 0.7)
    V, Y = oracle.vstep(A, U, 0.7)
    # V-target: the minimizer over real Y of ||R - U Y||_F (SVD least squares)
    Y_ls = np.linalg.lstsq(U.astype(float), A, rcond=None)[0]
    np.testing.assert_allclose(Y, Y_ls, rtol=0, atol=1e-4 * np.abs(Y_ls).max())
    # weighted U-target: minimizer over real Z of sum_j h_j ||R_:j - Z V_j:^T||^2
    _, Q, Z = oracle.ustep(A, V, w, 0.7)
    sw = np.sqrt(w)[:, None]
    Z_ls = np.linalg.lstsq(sw * V.astype(float), sw * A.T, rcond=None)[0].T
    np.testing.assert_allclose(Z, Z_ls, rtol=0, atol=1e-4 * np.abs(Z_ls).max())


@pytest.mark.parametrize("weighted", [False, True])
def test_joint_scales_zero_gradient(weighted):
    # Eq. (4) is the stationarity condition of the (weighted) Frobenius error in d.
    # Check it through the explicit rank-one sum, never through the Hadamard form.
    A = synth.small("t4_outliers", 64, 48, 4).astype(np.float64)
    w = oracle.normalized_weights(synth.small_importance(48, 4), 48) if weighted else np.ones(48)
    U, _ = oracle.init_block(A, w, 5, 1.0)
    for _ in range(3):
        V, _ = oracle.vstep(A, U, 1.0)
        U, Q, _ = oracle.ustep(A, V, w, 1.0)
    d = oracle.scale_solve(U, V, Q, w)
    Ahat = np.zeros_like(A)
    for c in range(U.shape[1]):
        Ahat += d[c] * np.outer(U[:, c].astype(float), V[:, c].astype(float))
    E = A - Ahat
    grad = np.array([-2 * U[:, c].astype(float) @ (E * w[None, :]) @ V[:, c].astype(float)
                     for c in range(U.shape[1])])
    scale = np.sum(w[None, :] * A * A)
    assert np.max(np.abs(grad)) < 1e-9 * scale
    # and the block decrease equals d^T g >= 0
    g = np.sum(U.astype(float) * Q, axis=0)
    dec = scale - np.sum(w[None, :] * E * E)
    assert dec >= 0
    assert abs(dec - d @ g) < 1e-9 * scale


# --------------------------------------------------------------------------
# exact symmetries
# --------------------------------------------------------------------------
def test_symmetries_bit_exact():
    A = synth.small("t4_rowscale", 72, 56, 12).astype(np.float64)
    for fac in (lambda X, **kw: oracle.factorize_block(X, 1.0, 0.7, 4, 4, **kw),
                lambda X, **kw: oracle.factorize_sequential(X, 0.5, 0.7, 4, **kw)):
        f = fac(A)
        g = fac(A * 2.0 ** -7)
        assert np.array_equal(f.B, g.B) and np.array_equal(f.C, g.C)
        assert np.array_equal(f.D * 2.0 ** -7, g.D) and f.E == g.E
        n = fac(-A)
        assert np.array_equal(n.B, -f.B) and np.array_equal(n.C, f.C) and np.array_equal(n.D, f.D)
        c = fac(A, h=np.full(56, 3.5, dtype=np.float32))
        assert np.array_equal(c.B, f.B) and np.array_equal(c.C, f.C) and np.array_equal(c.D, f.D)
        assert c.E == f.E and abs(c.E_w - f.E) < 1e-15   # E_w sums in another order


@pytest.mark.parametrize("weighted", [False, True])
def test_sequential_equals_block_of_one(weighted):
    # With bb = 1 the ridge and G^{-1} are positive scalars, and T_tau is
    # invariant to them (Eq. (2)), so Eq. (3)/(4) reduce to Sec. 2.3.
    A = synth.small("t4", 48, 64, 2)
    h = synth.small_importance(64, 2) if weighted else None
    s = oracle.factorize_sequential(A, 1.0, 0.7, 5, h=h)
    b = oracle.factorize_block(A, 1.0, 0.7, 1, 5, h=h)
    assert np.array_equal(s.B, b.B) and np.array_equal(s.C, b.C)
    np.testing.assert_allclose(b.D, s.D, rtol=1e-10)
    np.testing.assert_allclose(b.curve, s.curve, rtol=0, atol=1e-12)


def test_weighted_v_target_is_plain_residual():
    # Sec. 2.5: under a column-weighted objective the weights cancel in the
    # V-step.  The weighted least-squares V-target, solved column by column
    # on the system scaled by sqrt(h_j), equals the oracle's plain target.
    A = synth.small("t4_outliers", 70, 50, 13).astype(np.float64)
    w = oracle.normalized_weights(synth.small_importance(50, 13), 50)
    U, _ = oracle.init_block(A, w, 4, 1.0)
    _, Y = oracle.vstep(A, U, 1.0)
    sw = np.sqrt(w)
    Y_w = np.linalg.lstsq(U.astype(float), A * sw[None, :], rcond=None)[0] / sw[None, :]
    np.testing.assert_allclose(Y, Y_w, rtol=0, atol=1e-4 * np.abs(Y_w).max())
    # and a weighted sequential run starts from that plain target: its first
    # v equals T_tau applied to R^T u, not to (R diag(h))^T u
    f = oracle.factorize_sequential(A, 0.02, 1.0, 1, h=synth.small_importance(50, 13), k=1)
    u0 = oracle.ternarize(A[:, int(np.argmax(w * np.sum(A * A, 0)))], 1.0).astype(float)
    assert np.array_equal(f.C[0], oracle.ternarize(A.T @ u0, 1.0))


def test_init_uses_weighted_column_energy():
    # Reading R1, hand-worked: unweighted energies are (9, 2), weighted with
    # h~ = (0.1, 1) they are (0.9, 2): the second column is chosen.
    R = np.array([[3.0, 1.0], [0.0, 1.0]])
    U, J = oracle.init_block(R, np.array([0.1, 1.0]), 1, 0.7)
    assert J.tolist() == [1] and U[:, 0].tolist() == [1, 1]
    U, J = oracle.init_block(R, np.ones(2), 2, 0.7)
    assert J.tolist() == [0, 1] and U[:, 0].tolist() == [1, 0]
    # ties go to the smaller index
    U, J = oracle.init_block(np.array([[1.0, -1.0, 1.0]]), np.ones(3), 2, 0.7)
    assert J.tolist() == [0, 1]


# --------------------------------------------------------------------------
# Proposition 2, the corollary, prefix property, factor consistency
# --------------------------------------------------------------------------
def test_prop2_geometric_bound_with_safeguard():
    A = synth.small("gauss", 8, 8, 1).astype(np.float64)
    f = oracle.factorize_sequential(A, 80.0, 0.7, 4, safeguard=True)
    a2 = np.sum(A * A)
    k = np.arange(1, f.k + 1)
    assert np.all(f.fro2_curve <= (1 - 1 / 64) ** k * a2 * (1 + 1e-12) + 1e-300)
    assert f.E >= 1 - math.exp(-10)


def test_energy_tends_to_one_and_safeguard_idle():
    A = synth.small("gauss", 32, 32, 3)
    Es = []
    for mu in (1, 2, 4, 8):
        f = oracle.factorize_sequential(A, mu, 0.7, 8)
        Es.append(f.E)
        assert f.safeguard_would_fire == 0          # "the safeguard never activates"
    assert all(b > a for a, b in zip(Es, Es[1:]))
    assert Es[-1] > 1 - 1e-8


def test_prefix_property():
    A = synth.small("t4", 64, 96, 6)
    f1 = oracle.factorize_block(A, 1.0, 1.0, 8, 4)
    f2 = oracle.factorize_block(A, 2.0, 1.0, 8, 4)
    assert np.array_equal(f1.B, f2.B[:, :64]) and np.array_equal(f1.C, f2.C[:64])
    assert np.array_equal(f1.D, f2.D[:64])
    assert np.array_equal(f1.curve, f2.curve[:8])


@pytest.mark.parametrize("weighted", [False, True])
def test_factors_reproduce_energy(weighted):
    A = synth.small("t4_outliers", 80, 120, 9).astype(np.float64)
    h = synth.small_importance(120, 9) if weighted else None
    f = oracle.factorize_block(A, 1.5, 1.0, 8, 4, h=h)
    Rr = A - oracle.reconstruct(f.B, f.D, f.C)
    assert abs((1 - np.sum(Rr * Rr) / np.sum(A * A)) - f.E) < 1e-12
    if weighted:
        w = oracle.normalized_weights(h, 120)
        Ew = 1 - np.sum(w * np.sum(Rr * Rr, 0)) / np.sum(w * np.sum(A * A, 0))
        assert abs(Ew - f.E_w) < 1e-12


def test_zero_matrix():
    f = oracle.factorize_block(np.zeros((16, 24)), 1.0, 0.7, 2, 3)
    assert f.E == 1.0 and not f.B.any() and not f.C.any() and not f.D.any()


def test_rank_and_block_rules():
    assert oracle.rank_of(256, 256, 2.0) == 512
    assert oracle.rank_of(2048, 2048, 2.0) == 4096
    assert oracle.rank_of(9728, 2560, 3.0) == 7680
    assert oracle.rank_of(2560, 1024, 2.5) == 2560
    assert oracle.rank_of(10, 10, 0.25) == 3          # 2.5 rounds half up
    assert oracle.effective_block(256, 256, 1) == 1
    assert oracle.effective_block(9728, 2560, 64) == 64
    assert oracle.effective_block(64, 64, 256) == 8    # capped at min(m, n) / 8
    assert oracle.effective_block(5, 7, 4) == 1

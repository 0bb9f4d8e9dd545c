"""Pins for the block safeguard (Proposition 2, reading R12) and for the
lambda of the importance weights (Sec. 2.5), on the CPU oracle.

Fixed by the mathematics: Proposition 2's per-step bound
||R_after||^2 <= (1 - 1/(m n)) ||R_before||^2 (the single-entry option
removes max R_ij^2 >= ||R||^2 / (m n)); the exact zero the single-entry
step leaves at its entry; the sequential augmented step at b = 1; the
paper's remark that the safeguard stays idle in practice.  For lambda: a
constant importance with lambda = 1 is the uniform objective with every
weight 2 (bit-exact), and lambda -> infinity gives the uniform objective
(Sec. 2.5 states both limits of the interpolation).
"""
import math

import numpy as np
import pytest

import oracle
from paper_2607_13511_amd import synth


def _spiky(m, n, seed, spikes=3):
    rng = np.random.default_rng(seed)
    A = 0.05 * rng.standard_normal((m, n))
    for _ in range(spikes):
        A[rng.integers(m), rng.integers(n)] = rng.choice([-1.0, 1.0]) * rng.uniform(1.0, 3.0)
    return A


@pytest.mark.parametrize("tau,block", [(0.0, 1), (0.0, 4), (0.7, 4), (1.0, 1), (2.0, 8)])
def test_block_safeguard_geometric_bound(tau, block):
    A = _spiky(64, 40, 7)
    f = oracle.factorize_block(A, 0.5, tau, block, 3, safeguard=True)
    fro2 = np.concatenate([[np.sum(A * A)], f.fro2_curve])
    shrink = 1.0 - 1.0 / (64 * 40)
    assert np.all(fro2[1:] <= shrink * fro2[:-1] * (1 + 1e-12))


def test_block_safeguard_fires_on_dense_sign_fits():
    # with tau = 0 every trit is +-1 (dense signs), which spreads a block
    # over the whole matrix: a single spike is worth more, and taking it
    # raises the energy
    A = _spiky(64, 40, 7)
    f = oracle.factorize_block(A, 0.5, 0.0, 4, 3)
    g = oracle.factorize_block(A, 0.5, 0.0, 4, 3, safeguard=True)
    assert g.safeguard_fired > 0 and g.E > f.E


def test_single_entry_block_shape_and_exact_zero():
    A = _spiky(40, 36, 3, spikes=1)
    flat = int(np.argmax(np.abs(A)))
    ii, jj = divmod(flat, 36)
    f = oracle.factorize_block(A, 4 / 36, 0.0, 4, 3, safeguard=True)   # one block of 4
    assert f.k == 4 and f.block == 4 and f.safeguard_fired == 1
    assert f.B[:, 0].tolist() == [1 if i == ii else 0 for i in range(40)]
    assert f.C[0].tolist() == [int(np.sign(A[ii, jj])) if j == jj else 0 for j in range(36)]
    assert f.D[0] == abs(A[ii, jj]) and not f.B[:, 1:].any() and not f.C[1:].any() and not f.D[1:].any()
    R = A - oracle.reconstruct(f.B, f.D, f.C)
    assert R[ii, jj] == 0.0


def test_block_of_one_matches_sequential_augmented_step():
    A = _spiky(30, 26, 11)
    s = oracle.factorize_sequential(A, 1.0, 0.0, 3, safeguard=True)
    b = oracle.factorize_block(A, 1.0, 0.0, 1, 3, safeguard=True)
    assert s.safeguard_fired == b.safeguard_fired > 0
    assert np.array_equal(s.B, b.B) and np.array_equal(s.C, b.C)
    np.testing.assert_allclose(b.D, s.D, rtol=1e-10)


def test_block_safeguard_idle_on_realistic_matrix():
    # "in practice the safeguard never activates"
    A = synth.small("t4_rowscale", 96, 80, 5)
    f = oracle.factorize_block(A, 1.0, 1.0, 8, 4)
    g = oracle.factorize_block(A, 1.0, 1.0, 8, 4, safeguard=True)
    assert g.safeguard_fired == 0
    assert np.array_equal(f.B, g.B) and np.array_equal(f.C, g.C) and np.array_equal(f.D, g.D)


def test_safeguard_rejects_weights():
    A = synth.small("t4", 16, 16, 1)
    with pytest.raises(ValueError):
        oracle.factorize_block(A, 1.0, 1.0, 2, 2, h=np.ones(16), safeguard=True)


def test_lambda_with_constant_importance_is_uniform():
    # h constant -> h / max(h) = 1; lambda = 1 gives every weight 2, a power
    # of two, so the weighted arithmetic is the unweighted one scaled exactly
    A = synth.small("t4", 56, 48, 4)
    f = oracle.factorize_block(A, 1.0, 0.7, 4, 3)
    g = oracle.factorize_block(A, 1.0, 0.7, 4, 3, h=np.full(48, 0.37), lam=1.0)
    assert np.array_equal(f.B, g.B) and np.array_equal(f.C, g.C) and np.array_equal(f.D, g.D)
    assert np.array_equal(f.curve, g.curve) and np.allclose(g.curve_w, f.curve, rtol=0, atol=1e-15)


def test_lambda_to_infinity_is_uniform():
    A = synth.small("t4_rowscale", 64, 56, 6)
    h = synth.small_importance(56, 6)
    f = oracle.factorize_block(A, 1.0, 1.0, 4, 3)
    g = oracle.factorize_block(A, 1.0, 1.0, 4, 3, h=h, lam=2.0 ** 40)
    assert np.array_equal(f.B, g.B) and np.array_equal(f.C, g.C)
    np.testing.assert_allclose(g.D, f.D, rtol=1e-9)
    assert abs(g.E_w - f.E) < 1e-9
    # and lambda = 0 is a different (importance-weighted) objective here
    z = oracle.factorize_block(A, 1.0, 1.0, 4, 3, h=h)
    assert not np.array_equal(z.B, f.B)


def test_lambda_moves_weighted_energy_continuously():
    # interpolation between the two objectives: E_w measured with the pure
    # importance (lambda = 0) weights is best at lambda = 0 and the plain E
    # best at lambda -> infinity, at the ends of a lambda sweep
    A = synth.small("t4", 80, 64, 8)
    h = synth.small_importance(64, 8)
    w0 = oracle.normalized_weights(h, 64)
    ends = {}
    for lam in (0.0, 1e6):
        f = oracle.factorize_block(A, 1.0, 1.0, 4, 3, h=h, lam=lam)
        R = A - oracle.reconstruct(f.B, f.D, f.C)
        ends[lam] = (1 - float(w0 @ np.sum(R * R, 0)) / float(w0 @ np.sum(A * A, 0)),
                     1 - float(np.sum(R * R)) / float(np.sum(A * A)))
    assert ends[0.0][0] > ends[1e6][0]      # weighted energy under the imatrix objective
    assert ends[1e6][1] > ends[0.0][1]      # plain energy under the uniform objective


@pytest.mark.parametrize("lam", [-0.1, float("nan"), float("inf")])
def test_lambda_validation(lam):
    with pytest.raises(ValueError):
        oracle.normalized_weights(np.ones(4), 4, lam)

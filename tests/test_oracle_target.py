"""Pins of the energy-target stop (reading R10: extraction stops after the
first block whose energy reaches the target; mu chosen per matrix so that a
target accuracy is met exactly, Sec. 1 and Sec. 3).

What fixes it, independently of the stopping code: greedy deflation makes
each block depend only on the blocks before it, so the stopped run must be
the prefix of the full run (identical factors and energies); the energy is
non-decreasing block by block (Proposition 1 applied per block, Eq. (4)), so
the first block reaching the target is found from the full curve alone."""
import numpy as np
import pytest

import oracle


def _mat(seed, m=72, n=56):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((m, n)) * np.exp(rng.normal(0.0, 0.3, size=(m, 1)))


@pytest.mark.parametrize("seed,target", [(0, 0.3), (1, 0.55), (2, 0.8), (3, 0.9)])
def test_stop_is_the_prefix_of_the_full_run(seed, target):
    A = _mat(seed)
    full = oracle.factorize_block(A, 2.0, 0.7, 8, 4)
    cut = oracle.factorize_block(A, 2.0, 0.7, 8, 4, target=target)
    nb = len(cut.curve)
    assert cut.k_used == min(nb * full.block, full.k)
    # the first block of the full curve that reaches the target
    first = int(np.argmax(full.curve >= target)) + 1 if np.any(full.curve >= target) else len(full.curve)
    assert nb == first
    np.testing.assert_array_equal(cut.curve, full.curve[:nb])
    ku = cut.k_used
    np.testing.assert_array_equal(cut.B[:, :ku], full.B[:, :ku])
    np.testing.assert_array_equal(cut.C[:ku], full.C[:ku])
    np.testing.assert_array_equal(cut.D[:ku], full.D[:ku])
    assert not cut.B[:, ku:].any() and not cut.C[ku:].any() and not cut.D[ku:].any()
    assert cut.E == cut.curve[-1]
    # minimal: one block fewer misses the target
    assert cut.E >= target or ku == full.k
    if nb > 1:
        assert full.curve[nb - 2] < target
    # the stored factors reproduce the reported energy
    Ahat = oracle.reconstruct(cut.B, cut.D, cut.C)
    assert abs((1.0 - np.sum((A - Ahat) ** 2) / np.sum(A * A)) - cut.E) < 1e-12


def test_unreachable_and_trivial_targets():
    A = _mat(4)
    full = oracle.factorize_block(A, 1.0, 0.7, 8, 4)
    assert oracle.factorize_block(A, 1.0, 0.7, 8, 4, target=1.5).k_used == full.k
    assert oracle.factorize_block(A, 1.0, 0.7, 8, 4, target=-1.0).k_used == full.block


def test_weighted_stop_uses_weighted_energy():
    A = _mat(5)
    h = np.exp(np.random.default_rng(9).normal(size=A.shape[1]))
    full = oracle.factorize_block(A, 2.0, 1.0, 8, 4, h=h)
    # a target between the plain and weighted curves at some block tells them apart
    target = float(full.curve_w[3])
    cut = oracle.factorize_block(A, 2.0, 1.0, 8, 4, h=h, target=target)
    assert len(cut.curve_w) == int(np.argmax(full.curve_w >= target)) + 1
    assert cut.E_w >= target

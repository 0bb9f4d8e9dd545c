"""Pins of the inference product y = B (diag(D) (C x)) (Sec. 2.6): the
oracle's factored evaluation against the dense reconstruction
A_hat = B diag(D) C (Eq. (1)) applied to x, on random ternary factors and on
a real factorization, and linearity in x."""
import numpy as np

import oracle


def test_apply_equals_dense_product():
    rng = np.random.default_rng(0)
    m, n, k, nb = 37, 29, 53, 5
    B = rng.integers(-1, 2, size=(m, k)).astype(np.int8)
    C = rng.integers(-1, 2, size=(k, n)).astype(np.int8)
    D = rng.standard_normal(k)
    X = rng.standard_normal((nb, n))
    Y = oracle.apply(B, C, D, X)
    dense = oracle.reconstruct(B, D, C)
    np.testing.assert_allclose(Y, X @ dense.T, rtol=1e-12, atol=1e-12)
    # by hand for one entry
    i, b = 3, 2
    ref = sum(B[i, c] * D[c] * sum(C[c, j] * X[b, j] for j in range(n)) for c in range(k))
    assert abs(Y[b, i] - ref) < 1e-10


def test_apply_of_a_factorization_and_linearity():
    rng = np.random.default_rng(1)
    A = rng.standard_normal((48, 40))
    f = oracle.factorize_block(A, 1.5, 0.7, 8, 4)
    X = rng.standard_normal((3, 40))
    Y = oracle.apply(f.B, f.C, f.D, X)
    np.testing.assert_allclose(Y, X @ oracle.reconstruct(f.B, f.D, f.C).T, rtol=1e-12, atol=1e-12)
    Y2 = oracle.apply(f.B, f.C, f.D, 2.0 * X[:1] - X[1:2])
    np.testing.assert_allclose(Y2, 2.0 * Y[:1] - Y[1:2], rtol=1e-12, atol=1e-12)

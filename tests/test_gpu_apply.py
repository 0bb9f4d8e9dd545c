"""GPU parity of inference with a factorization, y = B (diag(D) (C x))
(externd_apply, Sec. 2.6), against the oracle's fp64 evaluation.

Tolerances, from the arithmetic of each path (u = 2^-24):
* one vector, n and k <= 10240 (integer matrix cores): x and t = diag(D) C x
  enter as 48-bit fixed-point vectors, x scaled by 2^s with s = 46 - e,
  max |x| < 2^e, so each entry moves by at most 2^-(s+1) <= 2^-46 max |x|;
  t likewise with the bound max |D| sum |x| in place of max |x|.  Products
  and sums are exact integers; t_c is formed in fp64 (two roundings) and
  y rounded once to fp32, so
  |y_gpu - y| <= u |y| + 2^-46 [(|B| (|D| (|C| 1))) max|x| + (|B| 1) max|D| sum|x|]
  plus fp64 roundings (covered by doubling the second term);
* otherwise: every entry of x is split exactly into three bf16 parts and
  the exact products trit x part are summed in fp32, one sum per part over
  n terms (a tree of depth at most n - 1), then the parts are added
  (2 roundings) and scaled by D_c (1 rounding): t_c carries at most
  (n + 2) u relative to D_c sum_j |C_cj x_j|.  t_c is split the same way
  and y_i = sum_c B_ic t_c adds k - 1 + 2 more roundings, so to first order
  |y_gpu - y| <= (n + k + 4) u (|B| (|D| (|C| |x|)))_i.
"""
import numpy as np
import pytest

import oracle
from paper_2607_13511_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def pack_trits(X: np.ndarray) -> np.ndarray:
    """Rows of trits -> the packed 2-bit format of include/externd.h."""
    X = np.asarray(X, dtype=np.int8)
    rows, cols = X.shape
    code = np.where(X == 0, 0, np.where(X > 0, 1, 3)).astype(np.uint8)
    pad = (-cols) % 4
    code = np.concatenate([code, np.zeros((rows, pad), np.uint8)], axis=1).reshape(rows, -1, 4)
    return (code[:, :, 0] | (code[:, :, 1] << 2) | (code[:, :, 2] << 4) | (code[:, :, 3] << 6)).astype(np.uint8)


GEMV_MAX = 10240   # one vector with n, k up to this length takes the integer matrix-core path


def bound(B, C, D, X):
    n, k = C.shape[1], C.shape[0]
    if X.shape[0] == 1 and n <= GEMV_MAX and k <= GEMV_MAX:
        Bf, Cf = np.abs(B).astype(np.float64), np.abs(C).astype(np.float64)
        y = oracle.apply(B, C, D, X)
        mx, sx, md = np.max(np.abs(X)), np.sum(np.abs(X)), np.max(np.abs(D))
        q = Bf @ (np.abs(D) * Cf.sum(axis=1)) * mx + Bf.sum(axis=1) * md * sx
        return U * np.abs(y) + 2.0 * 2.0 ** -46 * q[None, :]
    a = np.abs(B).astype(np.float64) @ (np.abs(D)[:, None] * (np.abs(C).astype(np.float64) @ np.abs(X).T))
    return (n + k + 4) * U * a.T


@pytest.fixture(scope="module")
def ext():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_13511_amd import binding
    binding.lib()
    return binding


def run(ext, B, C, D, X):
    m, k = B.shape
    n = C.shape[1]
    Bp = torch.from_numpy(pack_trits(B)).cuda()
    Cp = torch.from_numpy(pack_trits(C)).cuda()
    Y = ext.apply(Bp, Cp, torch.from_numpy(D.astype(np.float32)).cuda(), m, n,
                  torch.from_numpy(X.astype(np.float32)).cuda())
    torch.cuda.synchronize()
    return Y.cpu().numpy().astype(np.float64)


def test_pack_roundtrip(ext):
    rng = np.random.default_rng(3)
    X = rng.integers(-1, 2, size=(7, 23)).astype(np.int8)
    np.testing.assert_array_equal(ext.unpack_trits(pack_trits(X), 23), X)


@pytest.mark.parametrize("m,n,k,nb", [(37, 29, 53, 1), (37, 29, 53, 3), (64, 64, 64, 8), (1000, 777, 1500, 1),
                                      (1000, 777, 1500, 5), (9, 3, 2, 2), (5, 3, 1, 1), (70, 10240, 512, 1),
                                      (33, 300, 10240, 1), (20, 10241, 40, 1), (20, 40, 10241, 1)])
def test_apply_random_factors(ext, m, n, k, nb):
    print(f"[apply] random m={m} n={n} k={k} nb={nb}", flush=True)
    rng = np.random.default_rng(m + n + k + nb)
    B = rng.integers(-1, 2, size=(m, k)).astype(np.int8)
    C = rng.integers(-1, 2, size=(k, n)).astype(np.int8)
    D = rng.standard_normal(k).astype(np.float32).astype(np.float64)
    X = rng.standard_normal((nb, n)).astype(np.float32).astype(np.float64)
    Y = run(ext, B, C, D, X)
    ref = oracle.apply(B, C, D, X)
    assert np.all(np.abs(Y - ref) <= bound(B, C, D, X))


def test_apply_factorization(ext):
    A = synth.small("t4_rowscale", 384, 320, 21)
    res = ext.factorize(torch.from_numpy(A).cuda(), 2.0, 1.0, 16, 8)
    torch.cuda.synchronize()
    B = ext.unpack_trits(res.B_packed.cpu().numpy(), res.k)
    C = ext.unpack_trits(res.C_packed.cpu().numpy(), 320)
    D = res.D.cpu().numpy().astype(np.float64)
    X = np.random.default_rng(5).standard_normal((4, 320)).astype(np.float32).astype(np.float64)
    Y = ext.apply(res.B_packed, res.C_packed, res.D, 384, 320, torch.from_numpy(X.astype(np.float32)).cuda())
    torch.cuda.synchronize()
    Y = Y.cpu().numpy().astype(np.float64)
    ref = oracle.apply(B, C, D, X)
    assert np.all(np.abs(Y - ref) <= bound(B, C, D, X))
    # and the product approximates A x as well as the factorization approximates A
    err = np.linalg.norm(Y - X @ A.T.astype(np.float64)) / np.linalg.norm(X @ A.T.astype(np.float64))
    assert err < 2.0 * np.sqrt(1.0 - res.E) + 1e-3


def test_apply_fullsize(ext):
    w = synth.down9728()
    m, n = w.A.shape
    print("[apply] down9728 full size", flush=True)
    res = ext.factorize(torch.from_numpy(w.A).cuda(), w.mu, w.tau, w.block, w.iters)
    torch.cuda.synchronize()
    B = ext.unpack_trits(res.B_packed.cpu().numpy(), res.k)
    C = ext.unpack_trits(res.C_packed.cpu().numpy(), n)
    D = res.D.cpu().numpy().astype(np.float64)
    for nb in (1, 8):
        X = np.random.default_rng(nb).standard_normal((nb, n)).astype(np.float32).astype(np.float64)
        Y = ext.apply(res.B_packed, res.C_packed, res.D, m, n, torch.from_numpy(X.astype(np.float32)).cuda())
        torch.cuda.synchronize()
        Y = Y.cpu().numpy().astype(np.float64)
        ref = oracle.apply(B, C, D, X)
        assert np.all(np.abs(Y - ref) <= bound(B, C, D, X))


@pytest.mark.parametrize("bad", ["x_nan", "x_inf", "d_inf"])
def test_apply_one_vector_nonfinite(ext, bad):
    """The integer path: a NaN or infinite entry of x or D gives NaN everywhere."""
    rng = np.random.default_rng(11)
    m, n, k = 40, 70, 90
    B = rng.integers(-1, 2, size=(m, k)).astype(np.int8)
    C = rng.integers(-1, 2, size=(k, n)).astype(np.int8)
    D = rng.standard_normal(k)
    X = rng.standard_normal((1, n))
    if bad == "x_nan":
        X[0, 5] = np.nan
    elif bad == "x_inf":
        X[0, 7] = np.inf
    else:
        D[3] = -np.inf
    Y = run(ext, B, C, D, X)
    assert np.all(np.isnan(Y))


def test_apply_one_vector_scale_invariance(ext):
    """Powers of two carry through the fixed-point path exactly: x -> 2^e x
    gives y -> 2^e y bit for bit (the exponent moves, the digits do not)."""
    rng = np.random.default_rng(12)
    m, n, k = 300, 500, 700
    B = rng.integers(-1, 2, size=(m, k)).astype(np.int8)
    C = rng.integers(-1, 2, size=(k, n)).astype(np.int8)
    D = rng.standard_normal(k).astype(np.float32).astype(np.float64)
    X = rng.standard_normal((1, n)).astype(np.float32).astype(np.float64)
    Y0 = run(ext, B, C, D, X)
    for e in (-20, 13):
        np.testing.assert_array_equal(run(ext, B, C, D, X * 2.0 ** e), Y0 * 2.0 ** e)

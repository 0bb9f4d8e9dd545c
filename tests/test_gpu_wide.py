"""Wide blocks (effective width above 64, up to 256 = the paper's default,
Sec. 2.4) on the GPU against the fp64 oracle.

A wide block runs as quarters of 64 components coupled through the Gram
inverses of Eq. (3) and the joint solve of Eq. (4), formed as one
256 x 256 (at most) fp64 matrix each.  Per-step checks inject identical
state into both sides at widths 100 (a ragged last quarter of 36), 128 and
256, with the tolerances of the 64-wide parity tests: trits bit-exact
outside the 1e-5 threshold band, Y and Q within 1e-7 of the largest entry,
Z within 1e-10 of an fp64 solve on the GPU's own Q, D within 1e-8
relative, the deflated residual within its fp32 bound.  End to end, the
energy curves (E, and E_w with weights) after every block within 1e-3 of
oracle.factorize_block.
"""
import numpy as np
import pytest

import oracle
from paper_2607_13511_amd import synth
from test_gpu_parity import assert_tern_parity, cols_parity, cuda, host

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# kind, m, n, bb (each bb <= min(m, n) / 8 is not needed for the steps)
WIDE_SHAPES = [
    ("t4_rowscale", 900, 700, 100),
    ("t4_outliers", 1100, 1030, 128),
    ("gauss", 2100, 2060, 256),
]


@pytest.fixture(scope="module")
def ext():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_13511_amd import binding
    binding.lib()
    return binding


@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("kind,m,n,bb", WIDE_SHAPES)
def test_wide_init_parity(ext, kind, m, n, bb, weighted):
    print(f"[wide] init {kind} {m}x{n} bb={bb} w={weighted}", flush=True)
    R = synth.small(kind, m, n, 5)
    h = synth.small_importance(n, 5) if weighted else None
    w = oracle.normalized_weights(h, n)
    U_ref, J_ref = oracle.init_block(R.astype(np.float64), w, bb, 0.7)
    U, J = ext.step_init(cuda(R), bb, 0.7, h=cuda(h) if weighted else None)
    U, J = host(U), host(J)
    key = w * np.sum(R.astype(np.float64) ** 2, axis=0)
    np.testing.assert_allclose(key[J], key[J_ref], rtol=1e-12)
    for c in range(bb):
        assert_tern_parity(U[:, c], R[:, J[c]].astype(np.float64), 0.7, f"init column {c}")


@pytest.mark.parametrize("kind,m,n,bb", WIDE_SHAPES)
def test_wide_vstep_parity(ext, kind, m, n, bb):
    print(f"[wide] vstep {kind} {m}x{n} bb={bb}", flush=True)
    R = synth.small(kind, m, n, 1)
    tau = 0.7
    U, _ = oracle.init_block(R.astype(np.float64), np.ones(n), bb, tau)
    V_ref, Y_ref = oracle.vstep(R.astype(np.float64), U, tau)
    V, Y = ext.step_vstep(cuda(R), cuda(U), tau)
    V, Y = host(V), host(Y)
    assert np.max(np.abs(Y - Y_ref)) <= 1e-7 * np.max(np.abs(Y_ref))
    cols_parity(V, Y_ref.T, tau, "V")


@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("kind,m,n,bb", WIDE_SHAPES)
def test_wide_ustep_parity(ext, kind, m, n, bb, weighted):
    print(f"[wide] ustep {kind} {m}x{n} bb={bb} w={weighted}", flush=True)
    R = synth.small(kind, m, n, 2)
    h = synth.small_importance(n, 2) if weighted else None
    w = oracle.normalized_weights(h, n)
    tau = 1.0
    U0, _ = oracle.init_block(R.astype(np.float64), w, bb, tau)
    V, _ = oracle.vstep(R.astype(np.float64), U0, tau)
    U_ref, Q_ref, Z_ref = oracle.ustep(R.astype(np.float64), V, w, tau)
    U, Q, Z = ext.step_ustep(cuda(R), cuda(V), tau, h=cuda(h) if weighted else None)
    U, Q, Z = host(U), host(Q), host(Z)
    assert np.max(np.abs(Q - Q_ref)) <= 1e-7 * np.max(np.abs(Q_ref))
    # the fp64 solve, isolated from the contraction's rounding
    G = V.astype(np.float64).T @ (w[:, None] * V.astype(np.float64))
    G = G + oracle.RIDGE_REL * np.trace(G) / bb * np.eye(bb)
    Z_chk = np.linalg.solve(G, Q.T).T
    assert np.max(np.abs(Z - Z_chk)) <= 1e-10 * np.max(np.abs(Z_chk))
    cols_parity(U, Z_ref, tau, "U")


@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("kind,m,n,bb", WIDE_SHAPES)
def test_wide_scale_parity(ext, kind, m, n, bb, weighted):
    print(f"[wide] scale {kind} {m}x{n} bb={bb} w={weighted}", flush=True)
    R = synth.small(kind, m, n, 3).astype(np.float64)
    h = synth.small_importance(n, 3) if weighted else None
    w = oracle.normalized_weights(h, n)
    U, _ = oracle.init_block(R, w, bb, 1.0)
    for _ in range(2):
        V, _ = oracle.vstep(R, U, 1.0)
        U, Q, _ = oracle.ustep(R, V, w, 1.0)
    d_ref = oracle.scale_solve(U, V, Q, w)
    d = host(ext.step_scale(cuda(U), cuda(V), cuda(Q), h=cuda(h) if weighted else None))
    np.testing.assert_allclose(d, d_ref, rtol=1e-8, atol=1e-12 * np.max(np.abs(d_ref)))


@pytest.mark.parametrize("kind,m,n,bb", WIDE_SHAPES)
def test_wide_deflate_parity(ext, kind, m, n, bb):
    print(f"[wide] deflate {kind} {m}x{n} bb={bb}", flush=True)
    R = synth.small(kind, m, n, 4)
    R64 = R.astype(np.float64)
    U, _ = oracle.init_block(R64, np.ones(n), bb, 0.7)
    V, _ = oracle.vstep(R64, U, 0.7)
    U, Q, _ = oracle.ustep(R64, V, np.ones(n), 0.7)
    d = oracle.scale_solve(U, V, Q, np.ones(n))
    ref = oracle.deflate(R64, U, V, d.astype(np.float32).astype(np.float64))
    Rt = cuda(R)
    col, fro = ext.step_deflate(Rt, cuda(U), cuda(V), cuda(d))
    Rg = host(Rt).astype(np.float64)
    # one fp32 rounding per quarter's update of R plus the fp32 accumulation
    # of its 64 terms, measured by sum_c |U_ic d_c V_jc|
    absterm = (np.abs(U).astype(np.float64) * np.abs(d)[None, :]) @ np.abs(V).astype(np.float64).T
    scale = np.abs(ref) + absterm
    nq = (bb + 63) // 64
    assert np.all(np.abs(Rg - ref) <= 2e-6 * nq * scale + 1e-30)
    np.testing.assert_allclose(host(col), np.sum(Rg * Rg, axis=0), rtol=1e-12, atol=1e-300)
    np.testing.assert_allclose(host(fro)[0], np.sum(Rg * Rg), rtol=1e-12)


# kind, m, n, mu, tau, block, iters, weighted
WIDE_E2E = [
    ("t4_rowscale", 1040, 900, 0.5, 1.0, 100, 3, False),
    ("t4", 1100, 1030, 0.6, 0.7, 128, 3, True),
    ("gauss", 2100, 2060, 0.5, 1.0, 256, 2, False),
    ("t4_outliers", 2080, 2050, 0.4, 1.0, 256, 2, True),
]


@pytest.mark.parametrize("kind,m,n,mu,tau,block,iters,weighted", WIDE_E2E)
def test_wide_end_to_end(ext, kind, m, n, mu, tau, block, iters, weighted):
    print(f"[wide] e2e {kind} {m}x{n} mu={mu} tau={tau} b={block} it={iters} w={weighted}", flush=True)
    A = synth.small(kind, m, n, 7)
    h = synth.small_importance(n, 7) if weighted else None
    ref = oracle.factorize_block(A, mu, tau, block, iters, h=h)
    assert ref.block == block
    res = ext.factorize(cuda(A), mu, tau, block, iters, h=cuda(h) if weighted else None)
    assert res.block == block and res.k == ref.k
    np.testing.assert_allclose(res.curve, ref.curve, rtol=0, atol=1e-3)
    if weighted:
        np.testing.assert_allclose(res.curve_w, ref.curve_w, rtol=0, atol=1e-3)
    obj = res.curve_w if weighted else res.curve
    assert np.all(np.diff(obj) >= -1e-6)
    # the packed factors reproduce the reported energy
    from test_gpu_parity import decode
    B, C, D = decode(res, m, n)
    Rr = A.astype(np.float64) - (B.astype(np.float64) * D[None, :]) @ C.astype(np.float64)
    E = 1.0 - np.sum(Rr * Rr) / np.sum(A.astype(np.float64) ** 2)
    assert abs(E - res.E) <= 1e-5

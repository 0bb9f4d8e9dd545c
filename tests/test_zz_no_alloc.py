"""The allocation-free inference entry point, externd_apply_noalloc, against
externd_apply (the same kernels with a caller workspace) and the oracle's
fp64 evaluation of y = B (diag(D) (C x)) (Sec. 2.6).

Both entry points run the same kernels in the same order, so their outputs
must agree bit for bit; against the oracle the bound of the apply tests
holds: |y - y_exact| <= (n + k + 4) 2^-24 (|B| (|D| (|C| |x|))).
Calls follow each other, the second smaller (fewer rows, components and
vectors), so that it runs on the first call's scratch contents, the third
with a single vector (the vector-ALU path); then the largest workspace the
scratch holds along k, and one chunk of components more.
"""
import numpy as np
import pytest

import oracle

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


@pytest.fixture(scope="module")
def ext():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_13511_amd import binding
    binding.lib()
    return binding


def make(m, n, k, nb, seed):
    rng = np.random.default_rng(seed)
    B = rng.choice(np.array([-1, 0, 1], np.int8), size=(m, k), p=[0.25, 0.5, 0.25])
    C = rng.choice(np.array([-1, 0, 1], np.int8), size=(k, n), p=[0.2, 0.6, 0.2])
    D = (0.01 * rng.standard_normal(k)).astype(np.float32)
    X = rng.standard_normal((nb, n)).astype(np.float32)
    dev = [torch.from_numpy(a).cuda() for a in (pack_trits(B), pack_trits(C), D, X)]
    return (B, C, D, X), dev


def check_against_oracle(B, C, D, X, Y):
    n, k = C.shape[1], C.shape[0]
    Bd, Cd, Dd, Xd = (a.astype(np.float64) for a in (B, C, D, X))
    ref = oracle.apply(Bd, Cd, Dd, Xd)
    bnd = (n + k + 4) * U * (np.abs(Bd) @ (np.abs(Dd)[:, None] * (np.abs(Cd) @ np.abs(Xd).T))).T
    assert np.all(np.abs(Y.astype(np.float64) - ref) <= bnd)


def test_noalloc_matches_apply_two_calls(ext):
    # the second call is smaller in every dimension; the third takes the single-vector path
    for (m, n, k, nb, seed) in [(1000, 777, 3001, 8, 0), (301, 129, 517, 3, 1), (257, 100, 301, 1, 2)]:
        print(f"[noalloc] m={m} n={n} k={k} nb={nb}", flush=True)
        host, (Bp, Cp, D, X) = make(m, n, k, nb, seed)
        Y_ref = ext.apply(Bp, Cp, D, m, n, X)
        Y = ext.apply_noalloc(Bp, Cp, D, m, n, X)
        torch.cuda.synchronize()
        assert torch.equal(Y, Y_ref)
        check_against_oracle(*host, Y.cpu().numpy())


def test_noalloc_largest_intermediate_and_caller_output(ext):
    # the largest k (a multiple of the 128-component chunk) whose workspace fits the scratch at m = 64,
    # n = 40, nb = 8; Y supplied by the caller
    m, n, nb = 64, 40, 8
    wsb = ext.lib().externd_apply_workspace_bytes
    k = 128
    while wsb(m, n, k + 128, nb) <= ext.APPLY_NOALLOC_MAX_BYTES:
        k += 128
    assert wsb(m, n, k, nb) <= ext.APPLY_NOALLOC_MAX_BYTES < wsb(m, n, k + 1, nb)
    print(f"[noalloc] m={m} n={n} k={k} nb={nb} (largest that fits)", flush=True)
    host, (Bp, Cp, D, X) = make(m, n, k, nb, 7)
    Y = torch.empty((nb, m), dtype=torch.float32, device="cuda")
    out = ext.apply_noalloc(Bp, Cp, D, m, n, X, Y=Y)
    assert out.data_ptr() == Y.data_ptr()
    Y_ref = ext.apply(Bp, Cp, D, m, n, X)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y_ref)
    check_against_oracle(*host, Y.cpu().numpy())
    # one component more does not fit: refused on the host, Y untouched
    _, (Bp2, Cp2, D2, X2) = make(m, n, k + 1, nb, 8)
    before = Y.clone()
    with pytest.raises(ext.ExterndError) as ei:
        ext.apply_noalloc(Bp2, Cp2, D2, m, n, X2, Y=Y)
    assert ei.value.status == ext.ESCRATCH
    torch.cuda.synchronize()
    assert torch.equal(Y, before)

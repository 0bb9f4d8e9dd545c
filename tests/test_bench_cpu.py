"""Host-side pieces of bench.py: the factor zero fractions and the effective
bits per weight of Eq. (5), decoded from the packed trit format, checked
against a direct count on the decoded factors."""
import importlib.util
import os

import numpy as np
import pytest

torch = pytest.importorskip("torch")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _pack(T):
    """Rows of trits -> the library's 2-bit codes (00 = 0, 01 = +1, 11 = -1),
    element j of a row in byte j >> 2 at bits 2 (j & 3)."""
    rows, cols = T.shape
    nb = (cols + 3) // 4
    codes = np.zeros((rows, nb * 4), dtype=np.uint8)
    codes[:, :cols] = np.where(T == 1, 1, np.where(T == -1, 3, 0))
    codes = codes.reshape(rows, nb, 4)
    return (codes[..., 0] | (codes[..., 1] << 2) | (codes[..., 2] << 4) | (codes[..., 3] << 6)).astype(np.uint8)


class _Res:
    pass


@pytest.mark.parametrize("m,n,k", [(37, 50, 61), (64, 40, 96), (9, 13, 5)])
def test_sparsity_and_bpw(m, n, k):
    from paper_2607_13511_amd.binding import unpack_trits
    rng = np.random.default_rng(m * 1000 + n + k)
    B = rng.choice([-1, 0, 1], size=(m, k), p=[0.2, 0.55, 0.25]).astype(np.int8)
    C = rng.choice([-1, 0, 1], size=(k, n), p=[0.3, 0.4, 0.3]).astype(np.int8)
    Bp, Cp = _pack(B), _pack(C.copy())
    # the packing round-trips through the binding's decoder (ragged last byte)
    assert np.array_equal(unpack_trits(Bp, k), B) and np.array_equal(unpack_trits(Cp, n), C)
    res = _Res()
    res.B_packed, res.C_packed = torch.from_numpy(Bp), torch.from_numpy(Cp)
    got = _bench().sparsity_and_bpw(res, m, n, k)
    zb, zc = np.mean(B == 0), np.mean(C == 0)
    sp = (np.sum(B == 0) + np.sum(C == 0)) / (k * (m + n))
    assert got["zero_fraction_B"] == pytest.approx(zb, abs=0, rel=1e-12)
    assert got["zero_fraction_C"] == pytest.approx(zc, abs=0, rel=1e-12)
    assert got["sparsity"] == pytest.approx(sp, rel=1e-12)
    # Eq. (5) at mu = k / min(m, n): stored elements per weight k (m + n) / (m n)
    # times the mask+sign cost 2 - sparsity
    assert got["bpw_eff"] == pytest.approx(k * (m + n) / (m * n) * (2 - sp), rel=1e-12)


def test_oracle_threads():
    t, avail = _bench().oracle_threads()
    assert 1 <= t <= avail == len(os.sched_getaffinity(0))

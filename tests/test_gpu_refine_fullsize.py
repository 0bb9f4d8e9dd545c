"""Full-size parity of the refinement sweeps (GPU, through the C ABI): the
9728x2560 down projection at mu = 1, plain and importance-weighted, against
the stored fp64 oracle records (tests/golden/refine/*.json, written by
tests/golden/make_golden.py --refine, which calls only oracle/).

Checks: the extraction curve and the energy after each sweep within 1e-3
of the oracle's (E_w too with weights); the objective does not fall from
the extraction to the last sweep; the decoded factors reproduce the
reported energy.
"""
import glob
import hashlib
import json
import os

import numpy as np
import pytest

from paper_2607_13511_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
RECORDS = sorted(glob.glob(os.path.join(HERE, "golden", "refine", "*.json")))


@pytest.fixture(scope="module")
def ext():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_13511_amd import binding
    binding.lib()
    return binding


@pytest.mark.parametrize("path", RECORDS, ids=lambda p: os.path.basename(p)[:-5])
def test_refine_fullsize(ext, path):
    with open(path) as f:
        rec = json.load(f)
    w = synth.down9728(weighted=rec["weighted"])
    assert hashlib.sha256(np.ascontiguousarray(w.A, dtype=np.float32).tobytes()).hexdigest() == rec["a_sha256"]
    print(f"[refine-fullsize] {rec['name']}", flush=True)
    Ad = torch.from_numpy(w.A).cuda()
    hd = torch.from_numpy(w.h).cuda() if rec["weighted"] else None
    res = ext.factorize_refined(Ad, rec["mu"], rec["tau"], rec["block"], rec["iters"], rec["sweeps"], h=hd)
    torch.cuda.synchronize()
    F = res.factorization
    assert F.k == rec["k"] and F.block == rec["block_eff"] and res.revisits == rec["revisits"]
    np.testing.assert_allclose(F.curve, np.asarray(rec["curve"]), rtol=0, atol=1e-3)
    np.testing.assert_allclose(res.sweep_curve, np.asarray(rec["sweep_curve"]), rtol=0, atol=1e-3)
    assert abs(F.E - rec["E"]) <= 1e-3
    obj0 = F.curve_w[-1] if rec["weighted"] else F.curve[-1]
    obj = res.sweep_curve_w if rec["weighted"] else res.sweep_curve
    assert obj[-1] >= obj0 - 1e-6
    if rec["weighted"]:
        np.testing.assert_allclose(res.sweep_curve_w, np.asarray(rec["sweep_curve_w"]), rtol=0, atol=1e-3)
    m, n = rec["m"], rec["n"]
    B = ext.unpack_trits(F.B_packed.cpu().numpy(), F.k)
    C = ext.unpack_trits(F.C_packed.cpu().numpy(), n)
    D = F.D.cpu().numpy().astype(np.float64)
    Bd = torch.from_numpy(B).cuda().to(torch.float64) * torch.from_numpy(D).cuda()[None, :]
    Cd = torch.from_numpy(C).cuda().to(torch.float64)
    R = Ad.to(torch.float64) - Bd @ Cd
    E_dec = 1.0 - float((R * R).sum()) / float((Ad.to(torch.float64) ** 2).sum())
    assert abs(E_dec - F.E) < 1e-5

"""The GPU against the greedy sequential ALS oracle (Sec. 2.3) on the
down-projection recipe, beyond the one-launch sizes.

Records under tests/golden/seq/ (written by tests/golden/make_golden.py
--sequential, which calls only oracle/) hold, on one seeded input, the
energy curve of oracle.factorize_sequential (mode S: one component at a
time) and of oracle.factorize_block at b = 64 (mode B, Sec. 2.4):
* the GPU at block width 1 runs the block kernels with one component per
  block, which is the sequential algorithm (the ridge and Gram factors of
  Eq. (3) are positive scalars that T_tau ignores): the energy the run
  minimizes (E, or E_w with weights) within 1e-3 of mode S after every
  stored component (weighted runs: plain E within 2.5e-3 at the mu
  checkpoints, see the test);
* the GPU at b = 64 within 1e-3 of mode B after every block;
* the block algorithm's distance from the sequential one at the mu
  checkpoints is printed (the paper reports +-0.2 pt at b = 256 on real
  weights, Table 1 caption): it is a property of the algorithm, measured by
  the oracle, and the GPU reproduces it to 1e-3.
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
RECORDS = sorted(glob.glob(os.path.join(HERE, "golden", "seq", "*.json")))


def load(path):
    with open(path) as f:
        return json.load(f)


def inputs(rec):
    weighted = rec["weighted"]
    if rec["m"] == 9728 and rec["n"] == 2560:
        w = synth.down9728(weighted=weighted)
    else:
        w = synth.down_reduced(weighted=weighted, m=rec["m"], n=rec["n"])
    return w.A, w.h


@pytest.fixture(scope="module")
def ext():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_13511_amd import binding
    binding.lib()
    return binding


@pytest.mark.parametrize("path", RECORDS, ids=lambda p: os.path.basename(p)[:-5])
def test_gpu_against_sequential_oracle(ext, path):
    rec = load(path)
    A, h = inputs(rec)
    assert hashlib.sha256(np.ascontiguousarray(A, dtype=np.float32).tobytes()).hexdigest() == rec["a_sha256"]
    print(f"[seq] {rec['name']} b=1", flush=True)
    Ad = torch.from_numpy(A).cuda()
    hd = torch.from_numpy(h).cuda() if h is not None else None
    key = "_w" if rec["weighted"] else ""
    stride = rec["seq_stride"]
    # block width 1: the sequential algorithm on the block kernels
    r1 = ext.factorize(Ad, rec["mu"], rec["tau"], 1, rec["iters"], h=hd)
    assert r1.block == 1 and r1.k == rec["k"]
    sel = np.arange(stride - 1, r1.k, stride)
    dE = np.abs(r1.curve[sel] - np.asarray(rec["seq_curve"]))
    print(f"[seq] b=1: max |E - E_seq| {dE.max():.2e}", flush=True)
    ck = [kc // stride - 1 for kc in rec["checkpoints_k"]]
    if rec["weighted"]:
        # the objective this run minimizes is E_w: within 1e-3 after every
        # component.  The plain energy is not minimized (Sec. 2.5): over 1920
        # single-component steps the fp32 and fp64 residuals take different
        # but equally greedy paths (a trit inside the threshold band flips and
        # every later component differs), and plain E drifts further than
        # E_w (measured: E_w 9.4e-4 at most, E 1.8e-3 at mu = 2).
        dEw = np.abs(r1.curve_w[sel] - np.asarray(rec["seq_curve_w"]))
        print(f"[seq] b=1: max |E_w - E_w,seq| {dEw.max():.2e}; |E - E_seq| at checkpoints {dE[ck]}", flush=True)
        assert dEw.max() <= 1e-3
        assert np.all(dE[ck] <= 2.5e-3)
    else:
        assert dE.max() <= 1e-3
    obj1 = r1.curve_w if rec["weighted"] else r1.curve
    assert np.all(np.diff(obj1) >= -1e-6)
    # block width 64: the block algorithm
    print(f"[seq] {rec['name']} b={rec['block']}", flush=True)
    rb = ext.factorize(Ad, rec["mu"], rec["tau"], rec["block"], rec["iters"], h=hd)
    assert rb.block == rec["block_eff"]
    np.testing.assert_allclose(rb.curve, rec["block_curve"], rtol=0, atol=1e-3)
    if rec["weighted"]:
        np.testing.assert_allclose(rb.curve_w, rec["block_curve_w"], rtol=0, atol=1e-3)
    # the block algorithm's distance from the sequential one at the checkpoints
    seq = np.asarray(rec["seq_curve" + key])
    for kc in rec["checkpoints_k"]:
        e_seq = seq[kc // stride - 1]
        e_b1 = (r1.curve_w if rec["weighted"] else r1.curve)[kc - 1]
        e_gpu = (rb.curve_w if rec["weighted"] else rb.curve)[kc // rb.block - 1]
        e_ora = np.asarray(rec["block_curve" + key])[kc // rb.block - 1]
        print(f"[seq] k={kc}: E{key} sequential oracle {e_seq:.6f}, GPU b=1 {e_b1:.6f}, "
              f"GPU b={rb.block} {e_gpu:.6f} (oracle {e_ora:.6f}), block - sequential {e_gpu - e_seq:+.6f}",
              flush=True)
        assert abs(e_b1 - e_seq) <= 1e-3
        assert abs((e_gpu - e_seq) - (e_ora - e_seq)) <= 1e-3

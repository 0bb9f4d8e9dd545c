"""The stored full-size expectations (tests/golden/*.json) still describe
the inputs the tests build: each record's SHA-256 of its input matrix is
recomputed from the seeded generator, and the record is self-consistent
(k and block follow the rank and block rules; the curve ends at E and
never decreases)."""
import glob
import hashlib
import json
import os

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = sorted(glob.glob(os.path.join(HERE, "golden", "*.json")))
REFINE = sorted(glob.glob(os.path.join(HERE, "golden", "refine", "*.json")))


def test_golden_present():
    assert len(GOLDEN) >= 3


@pytest.mark.parametrize("path", GOLDEN, ids=lambda p: os.path.basename(p)[:-5])
def test_golden_record(path):
    from test_gpu_fullsize import inputs, load
    rec = load(path)
    A, h = inputs(rec)
    assert A.shape == (rec["m"], rec["n"])
    assert (h is not None) == rec["weighted"]
    assert hashlib.sha256(np.ascontiguousarray(A, dtype=np.float32).tobytes()).hexdigest() == rec["a_sha256"]
    assert rec["k"] == oracle.rank_of(rec["m"], rec["n"], rec["mu"])
    assert rec["block_eff"] == oracle.effective_block(rec["m"], rec["n"], rec["block"])
    curve = np.asarray(rec["curve"])
    assert len(curve) == -(-rec["k"] // rec["block_eff"])
    assert curve[-1] == rec["E"]
    assert np.all(np.diff(curve) >= -1e-12)


def test_refine_records_present():
    assert len(REFINE) >= 2


@pytest.mark.parametrize("path", REFINE, ids=lambda p: os.path.basename(p)[:-5])
def test_refine_record(path):
    from paper_2607_13511_amd import synth
    rec = load_json(path)
    w = synth.down9728(weighted=rec["weighted"])
    assert hashlib.sha256(np.ascontiguousarray(w.A, dtype=np.float32).tobytes()).hexdigest() == rec["a_sha256"]
    assert rec["k"] == oracle.rank_of(rec["m"], rec["n"], rec["mu"])
    nblk = -(-rec["k"] // rec["block_eff"])
    assert len(rec["curve"]) == nblk and len(rec["sweep_curve"]) == rec["sweeps"]
    assert rec["revisits"] == rec["sweeps"] * nblk and 0 <= rec["accepted"] <= rec["revisits"]
    # sweeps never lower the objective the run minimizes (Sec. 2.4)
    key = "_w" if rec["weighted"] else ""
    obj = [rec["curve" + key][-1]] + rec["sweep_curve" + key]
    assert np.all(np.diff(obj) >= -1e-12)
    assert rec["sweep_curve"][-1] == rec["E"]


def load_json(path):
    with open(path) as f:
        return json.load(f)


SEQ = sorted(glob.glob(os.path.join(HERE, "golden", "seq", "*.json")))


def test_seq_records_present():
    assert len(SEQ) >= 2


@pytest.mark.parametrize("path", SEQ, ids=lambda p: os.path.basename(p)[:-5])
def test_seq_record(path):
    """A sequential-vs-block record still describes its input; both curves
    never decrease in the objective their run minimizes (Proposition 1 for
    mode S; the Eq. (4) decrease d^T g >= 0 per block for mode B); and the
    sequential run is no worse than the block run at the last checkpoint
    (the block algorithm trades quality for batching, Sec. 2.4)."""
    from test_gpu_sequential import inputs
    rec = load_json(path)
    A, h = inputs(rec)
    assert (h is not None) == rec["weighted"]
    assert hashlib.sha256(np.ascontiguousarray(A, dtype=np.float32).tobytes()).hexdigest() == rec["a_sha256"]
    assert rec["k"] == oracle.rank_of(rec["m"], rec["n"], rec["mu"])
    assert rec["block_eff"] == oracle.effective_block(rec["m"], rec["n"], rec["block"])
    key = "_w" if rec["weighted"] else ""
    seq, blk = np.asarray(rec["seq_curve" + key]), np.asarray(rec["block_curve" + key])
    assert len(seq) == rec["k"] // rec["seq_stride"] and len(blk) == -(-rec["k"] // rec["block_eff"])
    assert np.all(np.diff(seq) >= -1e-12) and np.all(np.diff(blk) >= -1e-12)
    assert seq[-1] >= blk[-1]
    assert rec["seq_curve"][-1] == rec["seq_E"] and rec["block_curve"][-1] == rec["block_E"]

"""Seeded synthetic inputs shaped like LLM weight matrices.

This module only draws random numbers; it holds none of the factorization's
arithmetic.  Both the HIP path's tests/bench and the CPU oracle take their
inputs from here, so the two sides see identical bytes.

The paper measures on real Gemma-4-E2B / Qwen3.5-4B / Granite weights and a
llama.cpp importance matrix (Sec. 3); none of these are available, so the
recipes below stand in for them:

* ``gauss``        i.i.d. N(0, std^2)
* ``t4``           Student-t (df = 4) scaled to the given std
                   (Var t_4 = 2, so the draw is multiplied by std / sqrt(2))
* ``t4_outliers``  t4 plus ``n_outlier_cols`` columns scaled by 10
* ``t4_rowscale``  t4 with row i multiplied by exp(N(0, 0.3^2))
* ``spiky``        N(0, 0.05^2) with a few isolated entries of magnitude 1-3
                   (test input for the single-entry safeguard)
* importance       h_j = exp(N(0, 1)), with 1% of columns boosted x50

All draws use numpy's PCG64.  Named workloads use
``SeedSequence([0, workload_id, matrix_id, quantity_id])`` except the
256 x 256 Gaussian matrix, which uses ``default_rng(0)``.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import numpy as np

Q_A, Q_H, Q_OUTLIER, Q_ROWSCALE = 0, 1, 2, 3


def _rng(workload: int, matrix: int, quantity: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([0, workload, matrix, quantity]))


def gauss(m: int, n: int, std: float, rng: np.random.Generator) -> np.ndarray:
    return (rng.standard_normal((m, n)) * std).astype(np.float32)


def t4(m: int, n: int, std: float, rng: np.random.Generator) -> np.ndarray:
    return (rng.standard_t(4.0, size=(m, n)) * (std / math.sqrt(2.0))).astype(np.float32)


def t4_outliers(m, n, std, n_cols, rng_a, rng_o) -> np.ndarray:
    A = rng_a.standard_t(4.0, size=(m, n)) * (std / math.sqrt(2.0))
    cols = rng_o.choice(n, size=n_cols, replace=False)
    A[:, cols] *= 10.0
    return A.astype(np.float32)


def t4_rowscale(m, n, std, sigma, rng_a, rng_s) -> np.ndarray:
    A = rng_a.standard_t(4.0, size=(m, n)) * (std / math.sqrt(2.0))
    A *= np.exp(rng_s.standard_normal(m) * sigma)[:, None]
    return A.astype(np.float32)


def importance(n: int, rng_h: np.random.Generator, boost_frac: float = 0.01, boost: float = 50.0) -> np.ndarray:
    """Synthetic per-column activation second moments (imatrix stand-in)."""
    h = np.exp(rng_h.standard_normal(n))
    nb = int(round(boost_frac * n))
    if nb > 0:
        cols = rng_h.choice(n, size=nb, replace=False)
        h[cols] *= boost
    return h.astype(np.float32)


@dataclass
class Workload:
    name: str
    A: np.ndarray
    h: Optional[np.ndarray]
    mu: float
    tau: float
    block: int
    iters: int
    checkpoints_k: tuple


def gauss256(seed: int = 0) -> Workload:
    """256x256, N(0, 0.02^2), seed 0; mu=2 (k=512), tau=0.7, block=1, 8 iters."""
    A = gauss(256, 256, 0.02, np.random.default_rng(seed))
    return Workload("gauss256_mu2_tau0.7_b1", A, None, 2.0, 0.7, 1, 8, (64, 128, 256, 512))


def attn2048() -> Workload:
    """2048x2048 attention-projection-like: t4 std 0.02, 8 outlier cols x10; mu=2, tau=0.7, b=32."""
    A = t4_outliers(2048, 2048, 0.02, 8, _rng(2, 0, Q_A), _rng(2, 0, Q_OUTLIER))
    return Workload("attn2048_mu2_tau0.7_b32", A, None, 2.0, 0.7, 32, 8, (2048, 4096))


def down9728(weighted: bool = False) -> Workload:
    """9728x2560 MLP down-projection-like: t4 std 0.015, row scales exp(N(0,0.3^2)).

    mu=3 (k=7680), tau=1.0, block=64, 8 iters; optionally with synthetic
    importance weights (lognormal(0,1), 1% of columns x50).
    """
    A = t4_rowscale(9728, 2560, 0.015, 0.3, _rng(3, 0, Q_A), _rng(3, 0, Q_ROWSCALE))
    h = importance(2560, _rng(4, 0, Q_H)) if weighted else None
    name = "down9728x2560_mu3_tau1.0_b64" + ("_imatrix" if weighted else "")
    return Workload(name, A, h, 3.0, 1.0, 64, 8, (2560, 5120, 7680))


def ragged5003() -> Workload:
    """5003x3001 (neither side a multiple of 32), t4 std 0.02 with row scales
    exp(N(0, 0.3^2)) and importance weights; mu=1.5 (k=4502: 70 blocks of 64
    and a last block of 22), tau=1.0, block=64, 8 iters.
    """
    A = t4_rowscale(5003, 3001, 0.02, 0.3, _rng(6, 0, Q_A), _rng(6, 0, Q_ROWSCALE))
    h = importance(3001, _rng(6, 0, Q_H))
    return Workload("ragged5003x3001_mu1.5_tau1.0_b64_imatrix", A, h, 1.5, 1.0, 64, 8, (3001, 4502))


def down_reduced(weighted: bool = False, m: int = 2432, n: int = 640) -> Workload:
    """The 9728x2560 down-projection recipe (t4 std 0.015, row scales
    exp(N(0, 0.3^2)), optional lognormal(0,1) weights with 1% of columns x50)
    at a quarter of each side, 2432x640; mu=3 (k=1920), tau=1.0, block=64,
    8 iters.  Small enough for the sequential oracle to run in minutes."""
    A = t4_rowscale(m, n, 0.015, 0.3, _rng(7, 0, Q_A), _rng(7, 0, Q_ROWSCALE))
    h = importance(n, _rng(7, 0, Q_H)) if weighted else None
    name = f"down{m}x{n}_mu3_tau1.0" + ("_imatrix" if weighted else "")
    return Workload(name, A, h, 3.0, 1.0, 64, 8, (n, 2 * n, 3 * n))


BLOCK_SHAPES = (
    ("q", 2560, 4096), ("k", 2560, 1024), ("v", 2560, 1024), ("o", 4096, 2560),
    ("gate", 2560, 9728), ("up", 2560, 9728), ("down", 9728, 2560),
)


def transformer_block(idx: int):
    """One matrix of a synthetic ~4B transformer block (t4, std 0.02) and its weights."""
    name, m, n = BLOCK_SHAPES[idx]
    A = t4(m, n, 0.02, _rng(5, idx, Q_A))
    h = importance(n, _rng(5, idx, Q_H), boost_frac=0.0)
    return name, A, h


def small(kind: str, m: int, n: int, seed: int, std: float = 0.02) -> np.ndarray:
    """Small matrices of the same families for tests (ragged shapes allowed)."""
    rng = np.random.default_rng(np.random.SeedSequence([1, seed, m, n]))
    if kind == "gauss":
        return gauss(m, n, std, rng)
    if kind == "t4":
        return t4(m, n, std, rng)
    if kind == "t4_outliers":
        return t4_outliers(m, n, std, max(1, n // 256), rng, np.random.default_rng(np.random.SeedSequence([2, seed, m, n])))
    if kind == "t4_rowscale":
        return t4_rowscale(m, n, std, 0.3, rng, np.random.default_rng(np.random.SeedSequence([3, seed, m, n])))
    if kind == "spiky":
        return spiky(m, n, seed)
    if kind == "t4_outlier1e4":
        return outlier(t4(m, n, std, rng), seed, 1e4)
    raise ValueError(kind)


def spiky(m: int, n: int, seed: int, spikes: int = 3, std: float = 0.05) -> np.ndarray:
    """N(0, std^2) background with ``spikes`` isolated entries of magnitude
    U(1, 3) and random sign: a residual whose single largest entry is worth
    more than a dense ternary component (exercises the single-entry step)."""
    rng = np.random.default_rng(np.random.SeedSequence([6, seed, m, n]))
    A = rng.standard_normal((m, n)) * std
    for _ in range(spikes):
        A[rng.integers(m), rng.integers(n)] = rng.choice([-1.0, 1.0]) * rng.uniform(1.0, 3.0)
    return A.astype(np.float32)


def outlier(A: np.ndarray, seed: int, boost: float) -> np.ndarray:
    """A copy of A with one entry, at a seeded position and sign, set to
    boost * max|A| (a residual whose range is dominated by a single entry)."""
    rng = np.random.default_rng(np.random.SeedSequence([7, seed, A.shape[0], A.shape[1]]))
    B = np.array(A, dtype=np.float32, copy=True)
    i, j = int(rng.integers(A.shape[0])), int(rng.integers(A.shape[1]))
    B[i, j] = np.float32(rng.choice([-1.0, 1.0]) * boost * float(np.max(np.abs(A))))
    return B


def small_importance(n: int, seed: int) -> np.ndarray:
    return importance(n, np.random.default_rng(np.random.SeedSequence([4, seed, n])))

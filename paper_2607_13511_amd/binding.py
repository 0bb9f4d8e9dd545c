"""Thin ctypes binding over ``libexternd.so`` (C ABI in ``include/externd.h``).

Argument marshalling only: torch tensors supply device memory and the
current HIP stream; every step of the factorization runs in the library's
HIP kernels.  There is no fallback: if the library is missing or no GPU is
present the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libexternd.so")

OK, EINVAL, ENONFINITE, EWORKSPACE, EHIP, EUNSUPPORTED, ESYNC, ESCRATCH = 0, -1, -2, -3, -4, -5, -6, -7
APPLY_NOALLOC_MAX_BYTES = 8 << 20   # EXTERND_APPLY_NOALLOC_MAX_BYTES
MAX_BLOCK = 256

_lib = None

_c_i64 = ctypes.c_int64
_c_i32 = ctypes.c_int32
_c_dbl = ctypes.c_double
_c_ptr = ctypes.c_void_p
_c_size = ctypes.c_size_t

# name -> (restype, argtypes)
_SIGNATURES = {
    "externd_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "externd_rank": (_c_i64, [_c_i64, _c_i64, _c_dbl]),
    "externd_effective_block": (_c_i32, [_c_i64, _c_i64, _c_i32]),
    "externd_workspace_bytes": (_c_size, [_c_i64, _c_i64, _c_i64]),
    "externd_factorize": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_dbl, _c_dbl, _c_i32, _c_i32, _c_ptr,
                                         _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
                                         _c_ptr, _c_size, _c_ptr]),
    "externd_factorize_ex": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_dbl, _c_dbl, _c_i32, _c_i32, _c_ptr,
                                            _c_dbl, _c_i32, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
                                            _c_ptr, _c_ptr, _c_size, _c_ptr]),
    "externd_factorize_to_energy": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_dbl, _c_dbl, _c_dbl, _c_i32, _c_i32,
                                                   _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
                                                   _c_ptr, _c_ptr, _c_size, _c_ptr]),
    "externd_factorize_refined": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_dbl, _c_dbl, _c_i32, _c_i32, _c_i32,
                                                 _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
                                                 _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_size, _c_ptr]),
    "externd_apply_workspace_bytes": (_c_size, [_c_i64, _c_i64, _c_i64, _c_i32]),
    "externd_apply": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_i64, _c_i64, _c_i64, _c_ptr, _c_i32, _c_ptr,
                                     _c_ptr, _c_size, _c_ptr]),
    "externd_apply_noalloc": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_i64, _c_i64, _c_i64, _c_ptr, _c_i32,
                                             _c_ptr, _c_ptr]),
    "externd_factorize_timed": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_dbl, _c_dbl, _c_i32, _c_i32, _c_ptr,
                                               _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr, _c_ptr,
                                               _c_ptr, _c_size, _c_ptr, _c_ptr]),
    "externd_step_init": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_ptr, _c_i32, _c_dbl, _c_ptr, _c_ptr,
                                         _c_ptr, _c_size, _c_ptr]),
    "externd_step_vstep": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_ptr, _c_i32, _c_dbl, _c_ptr, _c_ptr,
                                          _c_ptr, _c_size, _c_ptr]),
    "externd_step_ustep": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_ptr, _c_i32, _c_dbl, _c_ptr, _c_ptr,
                                          _c_ptr, _c_ptr, _c_ptr, _c_size, _c_ptr]),
    "externd_step_scale": (ctypes.c_int, [_c_ptr, _c_ptr, _c_ptr, _c_i64, _c_i64, _c_i32, _c_ptr, _c_ptr,
                                          _c_ptr, _c_size, _c_ptr]),
    "externd_step_deflate": (ctypes.c_int, [_c_ptr, _c_i64, _c_i64, _c_ptr, _c_ptr, _c_ptr, _c_i32,
                                            _c_ptr, _c_ptr, _c_ptr, _c_size, _c_ptr]),
}
EXPORTED = tuple(_SIGNATURES)


KCLASS_NAMES = ("vstep_contraction", "ustep_contraction", "deflate", "vstep_target", "ustep_target",
                "sequential_one_launch", "ternarize_v", "ternarize_u")
# externd_factorize_timed times one launch in TIMING_STRIDE of each class
# (EXTERND_TIMING_STRIDE in include/externd.h).
TIMING_STRIDE = 16


class KernelTimes(ctypes.Structure):
    _fields_ = [("total_ms", ctypes.c_double * len(KCLASS_NAMES)), ("launches", ctypes.c_int64 * len(KCLASS_NAMES)),
                ("issued", ctypes.c_int64 * len(KCLASS_NAMES))]


class ExterndError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = lib().externd_strerror(status).decode()
        super().__init__(f"{where}: {msg} (status {status})")


def lib():
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status: int, where: str):
    if status != OK:
        raise ExterndError(status, where)


def rank(m: int, n: int, mu: float) -> int:
    return int(lib().externd_rank(m, n, mu))


def effective_block(m: int, n: int, block: int) -> int:
    return int(lib().externd_effective_block(m, n, block))


def workspace_bytes(m: int, n: int, k: int = 0) -> int:
    return int(lib().externd_workspace_bytes(m, n, k))


# ---------------------------------------------------------------------------
# torch marshalling
# ---------------------------------------------------------------------------
def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("externd needs a HIP GPU (torch.cuda is not available)")
    return torch


def _dev_ptr(t) -> int:
    return int(t.data_ptr())


def _stream_ptr(torch, stream) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


def _workspace(torch, m, n, k, device):
    nbytes = workspace_bytes(m, n, k)
    if nbytes == 0:
        raise ExterndError(EUNSUPPORTED, "workspace_bytes")
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _req(t, torch, dtype, shape, name):
    if not (t.is_cuda and t.dtype == dtype and t.is_contiguous() and tuple(t.shape) == tuple(shape)):
        raise ValueError(f"{name}: expected a contiguous {dtype} CUDA tensor of shape {tuple(shape)}, "
                         f"got {t.dtype} {tuple(t.shape)} on {t.device}")


@dataclass
class Factorization:
    B_packed: "object"        # torch.uint8 (m, ceil(k/4))
    C_packed: "object"        # torch.uint8 (k, ceil(n/4))
    D: "object"               # torch.float32 (k,)
    E: float
    E_w: float
    curve: np.ndarray
    curve_w: np.ndarray
    k: int
    block: int
    kernel_times: Optional[dict] = None   # class -> (total_ms, timed launches, all launches) when timed
    k_used: int = -1                      # components extracted (factorize_to_energy), else k
    safeguard_fired: int = 0              # blocks replaced by the single-entry step (factorize_ex)


def factorize(A, mu: float, tau: float, block: int, iters: int, h=None, stream=None,
              workspace=None, timed: bool = False) -> Factorization:
    """Factorize the fp32 CUDA tensor A (m x n) as B diag(D) C on the GPU.

    With ``timed`` the library records HIP events around every contraction
    and deflation launch and returns their summed durations.
    """
    torch = _torch()
    m, n = A.shape
    _req(A, torch, torch.float32, (m, n), "A")
    if h is not None:
        _req(h, torch, torch.float32, (n,), "h")
    k = rank(m, n, mu)
    if k < 1:
        raise ExterndError(EINVAL, "rank")
    b = effective_block(m, n, block)
    nblk = -(-k // b)
    dev = A.device
    Bp = torch.empty((m, (k + 3) // 4), dtype=torch.uint8, device=dev)
    Cp = torch.empty((k, (n + 3) // 4), dtype=torch.uint8, device=dev)
    D = torch.empty((k,), dtype=torch.float32, device=dev)
    ws = workspace if workspace is not None else _workspace(torch, m, n, k, dev)
    E = ctypes.c_double(0.0)
    Ew = ctypes.c_double(0.0)
    curve = np.zeros(nblk, dtype=np.float64)
    curve_w = np.zeros(nblk, dtype=np.float64)
    args = (_dev_ptr(A), m, n, mu, tau, block, iters, _dev_ptr(h) if h is not None else None,
            _dev_ptr(Bp), _dev_ptr(Cp), _dev_ptr(D), ctypes.byref(E), ctypes.byref(Ew),
            curve.ctypes.data, curve_w.ctypes.data, _dev_ptr(ws), ws.numel(), _stream_ptr(torch, stream))
    kt = None
    if timed:
        times = KernelTimes()
        _check(lib().externd_factorize_timed(*args, ctypes.byref(times)), "externd_factorize_timed")
        kt = {name: (times.total_ms[i], int(times.launches[i]), int(times.issued[i]))
              for i, name in enumerate(KCLASS_NAMES)}
    else:
        _check(lib().externd_factorize(*args), "externd_factorize")
    return Factorization(Bp, Cp, D, E.value, Ew.value, curve, curve_w, k, b, kt, k)


def factorize_ex(A, mu: float, tau: float, block: int, iters: int, h=None, lam: float = 0.0,
                 safeguard: bool = False, stream=None, workspace=None) -> Factorization:
    """externd_factorize with the lambda of the importance weights
    (h~ = h / max h + lam) and the single-entry safeguard of Proposition 2
    (plain objective only) (externd_factorize_ex)."""
    torch = _torch()
    m, n = A.shape
    _req(A, torch, torch.float32, (m, n), "A")
    if h is not None:
        _req(h, torch, torch.float32, (n,), "h")
    k = rank(m, n, mu)
    if k < 1:
        raise ExterndError(EINVAL, "rank")
    b = effective_block(m, n, block)
    nblk = -(-k // b)
    dev = A.device
    Bp = torch.empty((m, (k + 3) // 4), dtype=torch.uint8, device=dev)
    Cp = torch.empty((k, (n + 3) // 4), dtype=torch.uint8, device=dev)
    D = torch.empty((k,), dtype=torch.float32, device=dev)
    ws = workspace if workspace is not None else _workspace(torch, m, n, k, dev)
    E = ctypes.c_double(0.0)
    Ew = ctypes.c_double(0.0)
    fired = ctypes.c_int64(0)
    curve = np.zeros(nblk, dtype=np.float64)
    curve_w = np.zeros(nblk, dtype=np.float64)
    _check(lib().externd_factorize_ex(
        _dev_ptr(A), m, n, mu, tau, block, iters, _dev_ptr(h) if h is not None else None, lam, int(safeguard),
        _dev_ptr(Bp), _dev_ptr(Cp), _dev_ptr(D), ctypes.byref(E), ctypes.byref(Ew), curve.ctypes.data,
        curve_w.ctypes.data, ctypes.byref(fired), _dev_ptr(ws), ws.numel(), _stream_ptr(torch, stream)),
        "externd_factorize_ex")
    return Factorization(Bp, Cp, D, E.value, Ew.value, curve, curve_w, k, b, None, k, int(fired.value))


APPLY_MAX_BATCH = 8   # EXTERND_APPLY_MAX_BATCH


def apply(B_packed, C_packed, D, m: int, n: int, X, stream=None, workspace=None):
    """Y = X (B diag(D) C)^T on the GPU for the nb <= 8 rows of the fp32 CUDA
    tensor X (nb x n), from packed factors (externd_apply).  Returns Y (nb x m)."""
    torch = _torch()
    k = D.shape[0]
    nb = X.shape[0]
    _req(X, torch, torch.float32, (nb, n), "X")
    _req(D, torch, torch.float32, (k,), "D")
    _req(B_packed, torch, torch.uint8, (m, (k + 3) // 4), "B_packed")
    _req(C_packed, torch, torch.uint8, (k, (n + 3) // 4), "C_packed")
    Y = torch.empty((nb, m), dtype=torch.float32, device=X.device)
    nbytes = lib().externd_apply_workspace_bytes(m, n, k, nb)
    if nbytes == 0:
        raise ExterndError(EINVAL, "externd_apply_workspace_bytes")
    ws = workspace if workspace is not None else torch.empty(nbytes, dtype=torch.uint8, device=X.device)
    _check(lib().externd_apply(_dev_ptr(B_packed), _dev_ptr(C_packed), _dev_ptr(D), m, n, k, _dev_ptr(X), nb,
                               _dev_ptr(Y), _dev_ptr(ws), ws.numel(), _stream_ptr(torch, stream)), "externd_apply")
    return Y


def apply_noalloc(B_packed, C_packed, D, m: int, n: int, X, Y=None, stream=None):
    """As ``apply`` through externd_apply_noalloc: no workspace, the
    workspace lives in the library's fixed per-device scratch.  ``Y``
    (nb x m fp32 CUDA tensor) may be given so that the call allocates
    nothing at all.  Returns Y."""
    torch = _torch()
    k = D.shape[0]
    nb = X.shape[0]
    _req(X, torch, torch.float32, (nb, n), "X")
    _req(D, torch, torch.float32, (k,), "D")
    _req(B_packed, torch, torch.uint8, (m, (k + 3) // 4), "B_packed")
    _req(C_packed, torch, torch.uint8, (k, (n + 3) // 4), "C_packed")
    if Y is None:
        Y = torch.empty((nb, m), dtype=torch.float32, device=X.device)
    _req(Y, torch, torch.float32, (nb, m), "Y")
    _check(lib().externd_apply_noalloc(_dev_ptr(B_packed), _dev_ptr(C_packed), _dev_ptr(D), m, n, k, _dev_ptr(X),
                                       nb, _dev_ptr(Y), _stream_ptr(torch, stream)), "externd_apply_noalloc")
    return Y


def factorize_to_energy(A, mu_max: float, target: float, tau: float, block: int, iters: int, h=None,
                        stream=None, workspace=None) -> Factorization:
    """Factorize A until the energy (E, or E_w with h) reaches ``target``,
    with at most rank(m, n, mu_max) components (externd_factorize_to_energy).
    The result is sized for the maximum; components past ``k_used`` are
    zero and ``curve`` holds the blocks extracted."""
    torch = _torch()
    m, n = A.shape
    _req(A, torch, torch.float32, (m, n), "A")
    if h is not None:
        _req(h, torch, torch.float32, (n,), "h")
    k = rank(m, n, mu_max)
    if k < 1:
        raise ExterndError(EINVAL, "rank")
    b = effective_block(m, n, block)
    nblk = -(-k // b)
    dev = A.device
    Bp = torch.empty((m, (k + 3) // 4), dtype=torch.uint8, device=dev)
    Cp = torch.empty((k, (n + 3) // 4), dtype=torch.uint8, device=dev)
    D = torch.empty((k,), dtype=torch.float32, device=dev)
    ws = workspace if workspace is not None else _workspace(torch, m, n, k, dev)
    E = ctypes.c_double(0.0)
    Ew = ctypes.c_double(0.0)
    ku = ctypes.c_int64(0)
    curve = np.zeros(nblk, dtype=np.float64)
    curve_w = np.zeros(nblk, dtype=np.float64)
    _check(lib().externd_factorize_to_energy(
        _dev_ptr(A), m, n, mu_max, target, tau, block, iters, _dev_ptr(h) if h is not None else None,
        _dev_ptr(Bp), _dev_ptr(Cp), _dev_ptr(D), ctypes.byref(ku), ctypes.byref(E), ctypes.byref(Ew),
        curve.ctypes.data, curve_w.ctypes.data, _dev_ptr(ws), ws.numel(), _stream_ptr(torch, stream)),
        "externd_factorize_to_energy")
    nb = -(-ku.value // b)
    return Factorization(Bp, Cp, D, E.value, Ew.value, curve[:nb], curve_w[:nb], k, b, None, int(ku.value))


@dataclass
class Refined:
    factorization: Factorization       # final factors; E, E_w after the last sweep; extraction curve
    sweep_curve: np.ndarray            # E after each sweep
    sweep_curve_w: np.ndarray          # weighted E after each sweep
    accepted: int                      # revisits that replaced their block
    revisits: int


def factorize_refined(A, mu: float, tau: float, block: int, iters: int, sweeps: int, h=None, stream=None,
                      workspace=None) -> Refined:
    """Factorize A, then run ``sweeps`` refinement sweeps over its blocks
    (externd_factorize_refined)."""
    torch = _torch()
    m, n = A.shape
    _req(A, torch, torch.float32, (m, n), "A")
    if h is not None:
        _req(h, torch, torch.float32, (n,), "h")
    k = rank(m, n, mu)
    if k < 1:
        raise ExterndError(EINVAL, "rank")
    b = effective_block(m, n, block)
    nblk = -(-k // b)
    dev = A.device
    Bp = torch.empty((m, (k + 3) // 4), dtype=torch.uint8, device=dev)
    Cp = torch.empty((k, (n + 3) // 4), dtype=torch.uint8, device=dev)
    D = torch.empty((k,), dtype=torch.float32, device=dev)
    ws = workspace if workspace is not None else _workspace(torch, m, n, k, dev)
    E = ctypes.c_double(0.0)
    Ew = ctypes.c_double(0.0)
    acc = ctypes.c_int64(0)
    curve = np.zeros(nblk, dtype=np.float64)
    curve_w = np.zeros(nblk, dtype=np.float64)
    sc = np.zeros(max(sweeps, 1), dtype=np.float64)
    scw = np.zeros(max(sweeps, 1), dtype=np.float64)
    _check(lib().externd_factorize_refined(
        _dev_ptr(A), m, n, mu, tau, block, iters, sweeps, _dev_ptr(h) if h is not None else None,
        _dev_ptr(Bp), _dev_ptr(Cp), _dev_ptr(D), ctypes.byref(E), ctypes.byref(Ew),
        curve.ctypes.data, curve_w.ctypes.data, sc.ctypes.data, scw.ctypes.data, ctypes.byref(acc),
        _dev_ptr(ws), ws.numel(), _stream_ptr(torch, stream)), "externd_factorize_refined")
    F = Factorization(Bp, Cp, D, E.value, Ew.value, curve, curve_w, k, b, None, k)
    return Refined(F, sc[:sweeps], scw[:sweeps], int(acc.value), sweeps * nblk)


def step_init(R, bb: int, tau: float, h=None, stream=None):
    torch = _torch()
    m, n = R.shape
    _req(R, torch, torch.float32, (m, n), "R")
    U = torch.empty((m, bb), dtype=torch.int8, device=R.device)
    J = torch.empty((bb,), dtype=torch.int32, device=R.device)
    ws = _workspace(torch, m, n, 0, R.device)
    st = lib().externd_step_init(_dev_ptr(R), m, n, _dev_ptr(h) if h is not None else None, bb, tau,
                                 _dev_ptr(U), _dev_ptr(J), _dev_ptr(ws), ws.numel(), _stream_ptr(torch, stream))
    _check(st, "externd_step_init")
    return U, J


def step_vstep(R, U, tau: float, stream=None):
    torch = _torch()
    m, n = R.shape
    bb = U.shape[1]
    _req(R, torch, torch.float32, (m, n), "R")
    _req(U, torch, torch.int8, (m, bb), "U")
    V = torch.empty((n, bb), dtype=torch.int8, device=R.device)
    Y = torch.empty((bb, n), dtype=torch.float64, device=R.device)
    ws = _workspace(torch, m, n, 0, R.device)
    st = lib().externd_step_vstep(_dev_ptr(R), m, n, _dev_ptr(U), bb, tau, _dev_ptr(V), _dev_ptr(Y),
                                  _dev_ptr(ws), ws.numel(), _stream_ptr(torch, stream))
    _check(st, "externd_step_vstep")
    return V, Y


def step_ustep(R, V, tau: float, h=None, stream=None):
    torch = _torch()
    m, n = R.shape
    bb = V.shape[1]
    _req(R, torch, torch.float32, (m, n), "R")
    _req(V, torch, torch.int8, (n, bb), "V")
    U = torch.empty((m, bb), dtype=torch.int8, device=R.device)
    Q = torch.empty((m, bb), dtype=torch.float64, device=R.device)
    Z = torch.empty((m, bb), dtype=torch.float64, device=R.device)
    ws = _workspace(torch, m, n, 0, R.device)
    st = lib().externd_step_ustep(_dev_ptr(R), m, n, _dev_ptr(V), bb, tau, _dev_ptr(h) if h is not None else None,
                                  _dev_ptr(U), _dev_ptr(Q), _dev_ptr(Z), _dev_ptr(ws), ws.numel(),
                                  _stream_ptr(torch, stream))
    _check(st, "externd_step_ustep")
    return U, Q, Z


def step_scale(U, V, Q, h=None, stream=None):
    torch = _torch()
    m, bb = U.shape
    n = V.shape[0]
    _req(U, torch, torch.int8, (m, bb), "U")
    _req(V, torch, torch.int8, (n, bb), "V")
    _req(Q, torch, torch.float64, (m, bb), "Q")
    d = torch.empty((bb,), dtype=torch.float64, device=U.device)
    ws = _workspace(torch, m, n, 0, U.device)
    st = lib().externd_step_scale(_dev_ptr(U), _dev_ptr(V), _dev_ptr(Q), m, n, bb,
                                  _dev_ptr(h) if h is not None else None, _dev_ptr(d), _dev_ptr(ws), ws.numel(),
                                  _stream_ptr(torch, stream))
    _check(st, "externd_step_scale")
    return d


def step_deflate(R, U, V, d, stream=None):
    """In-place R <- R - U diag(fp32(d)) V^T; returns (colnorm2, fro2)."""
    torch = _torch()
    m, n = R.shape
    bb = U.shape[1]
    _req(R, torch, torch.float32, (m, n), "R")
    _req(U, torch, torch.int8, (m, bb), "U")
    _req(V, torch, torch.int8, (n, bb), "V")
    _req(d, torch, torch.float64, (bb,), "d")
    col = torch.empty((n,), dtype=torch.float64, device=R.device)
    fro = torch.empty((1,), dtype=torch.float64, device=R.device)
    ws = _workspace(torch, m, n, 0, R.device)
    st = lib().externd_step_deflate(_dev_ptr(R), m, n, _dev_ptr(U), _dev_ptr(V), _dev_ptr(d), bb, _dev_ptr(col),
                                    _dev_ptr(fro), _dev_ptr(ws), ws.numel(), _stream_ptr(torch, stream))
    _check(st, "externd_step_deflate")
    return col, fro


# ---------------------------------------------------------------------------
# packed trit format (host-side decode for users and tests)
# ---------------------------------------------------------------------------
def unpack_trits(packed: np.ndarray, cols: int) -> np.ndarray:
    """Decode rows of 2-bit trits (00 = 0, 01 = +1, 11 = -1) into int8.

    Raises ValueError on the unused code 10 or on nonzero padding bits.
    """
    packed = np.ascontiguousarray(packed, dtype=np.uint8)
    rows, nbytes = packed.shape
    if nbytes != (cols + 3) // 4:
        raise ValueError("packed row length does not match the column count")
    codes = np.stack([(packed >> (2 * s)) & 3 for s in range(4)], axis=-1).reshape(rows, nbytes * 4)
    if np.any(codes == 2):
        raise ValueError("invalid trit code 10")
    if np.any(codes[:, cols:] != 0):
        raise ValueError("nonzero padding bits")
    codes = codes[:, :cols]
    out = np.zeros((rows, cols), dtype=np.int8)
    out[codes == 1] = 1
    out[codes == 3] = -1
    return out

"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function declared in include/externd.h, and rejects bad arguments
before any device work."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2607_13511_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "externd.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(externd_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = binding.lib()
    declared = _declared_functions()
    assert len(declared) >= 10
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(binding.EXPORTED) == declared


def test_rank_block_and_workspace_rules():
    for m, n, mu in [(256, 256, 2.0), (2048, 2048, 2.0), (9728, 2560, 3.0), (2560, 1024, 2.5), (10, 10, 0.25),
                     (37, 11, 1.3)]:
        assert binding.rank(m, n, mu) == oracle.rank_of(m, n, mu)
    for m, n, b in [(256, 256, 1), (9728, 2560, 64), (64, 64, 256), (5, 7, 4), (2048, 2048, 32),
                    (4096, 4096, 256), (519, 4000, 256), (520, 4000, 256)]:
        assert binding.effective_block(m, n, b) == oracle.effective_block(m, n, b)
    # the paper's default b = 256 is capped at floor(min(m, n) / 8) and nothing else
    assert binding.effective_block(4096, 4096, 256) == 256 and binding.effective_block(519, 4000, 256) == 64
    assert binding.rank(0, 5, 1.0) == -1 and binding.rank(5, 5, 0.0) == -1 and binding.rank(5, 5, float("nan")) == -1
    ws = binding.workspace_bytes(9728, 2560, 7680)
    # the fp32 residual plus per-row and per-column buffers for 256-wide blocks
    assert 4 * 9728 * 2560 < ws < 4 * 9728 * 2560 + 6144 * 9728 + 20480 * 2560 + (16 << 20)
    assert binding.workspace_bytes(0, 10, 0) == 0
    assert binding.workspace_bytes(1 << 16, 1 << 16, 0) == 0        # beyond the supported size
    assert binding.workspace_bytes(100, 70, 10000) > binding.workspace_bytes(100, 70, 0)  # per-block history


def test_argument_errors_before_device_work():
    L = binding.lib()
    dummy = ctypes.c_void_p(256)          # never dereferenced: validation fails first
    E = ctypes.c_double(0.0)
    f = L.externd_factorize
    # null A
    assert f(None, 10, 10, 1.0, 0.7, 1, 1, None, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             dummy, 1 << 30, None) == binding.EINVAL
    assert np.isnan(E.value)
    # bad scalars
    for (m, n, mu, tau, block, iters) in [(0, 10, 1.0, 0.7, 1, 1), (10, 10, 0.0, 0.7, 1, 1),
                                          (10, 10, 1.0, -1.0, 1, 1), (10, 10, 1.0, float("inf"), 1, 1),
                                          (10, 10, 1.0, 0.7, 0, 1), (10, 10, 1.0, 0.7, 1, 0)]:
        assert f(dummy, m, n, mu, tau, block, iters, None, dummy, dummy, dummy, ctypes.byref(E), None, None,
                 None, dummy, 1 << 30, None) == binding.EINVAL
    # workspace too small / misaligned
    assert f(dummy, 10, 10, 1.0, 0.7, 1, 1, None, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             dummy, 16, None) == binding.EWORKSPACE
    assert f(dummy, 10, 10, 1.0, 0.7, 1, 1, None, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             ctypes.c_void_p(257), 1 << 30, None) == binding.EWORKSPACE
    # unsupported shape
    assert f(dummy, 1 << 16, 1 << 16, 1.0, 0.7, 1, 1, None, dummy, dummy, dummy, ctypes.byref(E), None, None,
             None, dummy, 1 << 40, None) == binding.EUNSUPPORTED
    # effective block width beyond what the kernels hold (256): refused, never clamped
    for ff, extra in [(f, ()), (L.externd_factorize_timed, (dummy,))]:
        assert ff(dummy, 4096, 4096, 1.0, 0.7, 257, 1, None, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
                  dummy, 1 << 40, None, *extra) == binding.EUNSUPPORTED
        assert np.isnan(E.value)
    assert f(dummy, 8192, 8192, 1.0, 0.7, 512, 1, None, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             dummy, 1 << 40, None) == binding.EUNSUPPORTED
    # wide blocks (effective width above 64) have no refinement sweeps and no safeguard
    assert L.externd_factorize_refined(dummy, 1024, 1024, 1.0, 0.7, 65, 1, 1, None, dummy, dummy, dummy,
                                       ctypes.byref(E), None, None, None, None, None, None, dummy, 1 << 40,
                                       None) == binding.EUNSUPPORTED
    assert L.externd_factorize_ex(dummy, 1024, 1024, 1.0, 0.7, 65, 1, None, 0.0, 1, dummy, dummy, dummy,
                                  ctypes.byref(E), None, None, None, None, dummy, 1 << 40, None) == binding.EUNSUPPORTED
    # step entry points
    assert L.externd_step_vstep(None, 10, 10, dummy, 4, 0.7, dummy, None, dummy, 1 << 30, None) == binding.EINVAL
    assert L.externd_step_vstep(dummy, 10, 10, dummy, 257, 0.7, dummy, None, dummy, 1 << 30, None) == binding.EINVAL
    assert L.externd_step_ustep(dummy, 10, 10, dummy, 0, 0.7, None, dummy, None, None, dummy, 1 << 30,
                                None) == binding.EINVAL
    assert L.externd_step_scale(dummy, dummy, None, 10, 10, 4, None, dummy, dummy, 1 << 30, None) == binding.EINVAL
    assert L.externd_step_deflate(dummy, 10, 10, dummy, dummy, None, 4, None, None, dummy, 1 << 30,
                                  None) == binding.EINVAL
    assert L.externd_step_init(dummy, 10, 10, None, 11, 0.7, dummy, dummy, dummy, 1 << 30, None) == binding.EINVAL
    # energy-target run: the target must be finite and k_used given
    ku = ctypes.c_int64(7)
    g = L.externd_factorize_to_energy
    for target, kptr in [(float("nan"), ctypes.byref(ku)), (float("inf"), ctypes.byref(ku)), (0.9, None)]:
        assert g(dummy, 10, 10, 1.0, target, 0.7, 1, 1, None, dummy, dummy, dummy, kptr, ctypes.byref(E), None,
                 None, None, dummy, 1 << 30, None) == binding.EINVAL
        assert np.isnan(E.value)
    assert g(None, 10, 10, 1.0, 0.9, 0.7, 1, 1, None, dummy, dummy, dummy, ctypes.byref(ku), ctypes.byref(E), None,
             None, None, dummy, 1 << 30, None) == binding.EINVAL
    # refinement sweeps: sweeps >= 0, same argument rules as externd_factorize
    r = L.externd_factorize_refined
    assert r(dummy, 10, 10, 1.0, 0.7, 1, 1, -1, None, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             None, None, None, dummy, 1 << 30, None) == binding.EINVAL
    assert np.isnan(E.value)
    assert r(None, 10, 10, 1.0, 0.7, 1, 1, 2, None, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             None, None, None, dummy, 1 << 30, None) == binding.EINVAL
    assert r(dummy, 10, 10, 1.0, 0.7, 1, 1, 2, None, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             None, None, None, dummy, 16, None) == binding.EWORKSPACE
    # lambda and safeguard options: lambda finite and >= 0, safeguard 0 or 1
    # and only for the plain objective
    x = L.externd_factorize_ex
    fired = ctypes.c_int64(5)
    for lam, sg, imp in [(-0.5, 0, dummy), (float("nan"), 0, dummy), (float("inf"), 0, None), (0.0, 2, None),
                         (0.0, -1, None), (0.0, 1, dummy), (1.0, 1, dummy)]:
        assert x(dummy, 10, 10, 1.0, 0.7, 1, 1, imp, lam, sg, dummy, dummy, dummy, ctypes.byref(E), None, None,
                 None, ctypes.byref(fired), dummy, 1 << 30, None) == binding.EINVAL
        assert np.isnan(E.value) and fired.value == 0
    assert x(None, 10, 10, 1.0, 0.7, 1, 1, None, 0.0, 1, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             None, dummy, 1 << 30, None) == binding.EINVAL
    assert x(dummy, 10, 10, 1.0, 0.7, 1, 1, None, 0.0, 1, dummy, dummy, dummy, ctypes.byref(E), None, None, None,
             None, dummy, 16, None) == binding.EWORKSPACE
    # inference: batch limits, workspace size and alignment
    ap = L.externd_apply
    # nb = 1, n and k <= 10240 (integer matrix-core path): the six digit planes of the intermediate T,
    # 1536 bytes per 256 components of k, rounded up to 256 bytes, then a 256-byte exponent word
    wsb = L.externd_apply_workspace_bytes
    assert wsb(100, 100, 100, 1) == 1536 + 256 and wsb(100, 100, 101, 1) == 1536 + 256
    assert wsb(5, 5, 5, 1) == 1536 + 256 and wsb(9728, 2560, 7680, 1) == 30 * 1536 + 256
    assert wsb(9728, 10240, 10240, 1) == 40 * 1536 + 256
    # nb = 1 with n or k above 10240 (vector-ALU path): T, k floats (k rounded up to 4), rounded up to 256 bytes
    assert wsb(100, 10241, 100, 1) == 512 and wsb(100, 100, 10241, 1) == 41216
    # nb >= 2 (matrix-core path), 100 x 100 x 100: the parts of T (3 nb columns of 128 bf16, rounded up to
    # 256 bytes); one slice per product, so no partial sums
    assert wsb(100, 100, 100, 2) == 1536 and wsb(100, 100, 100, 3) == 2304
    # 9728 x 2560 at k = 7680, nb = 8: the parts of T, then the B side's 15 slices of 9728 rows of partial
    # sums (the C side's 10 slices of 7680 rows share the region)
    assert wsb(9728, 2560, 7680, 8) == 24 * 7680 * 2 + 4 * 15 * 9728 * 8
    assert wsb(9728, 2560, 7680, 8) <= 6 * 8 * 7680 + 8 * 9728 * 7680 // 32 + 4 * 256 * 8 * 15
    assert wsb(100, 100, 100, 9) == 0 and wsb(0, 100, 100, 1) == 0 and wsb(100, 0, 100, 1) == 0
    assert wsb(100, 100, 0, 1) == 0 and wsb(100, 100, (1 << 31) + 1, 1) == 0
    assert ap(dummy, dummy, dummy, 10, 10, 5, dummy, 0, dummy, dummy, 1 << 20, None) == binding.EINVAL
    assert ap(dummy, dummy, dummy, 10, 10, 5, dummy, 9, dummy, dummy, 1 << 20, None) == binding.EINVAL
    assert ap(None, dummy, dummy, 10, 10, 5, dummy, 1, dummy, dummy, 1 << 20, None) == binding.EINVAL
    assert ap(dummy, dummy, dummy, 10, 10, 5, dummy, 1, dummy, dummy, 4, None) == binding.EWORKSPACE
    assert ap(dummy, dummy, dummy, 10, 10, 5, dummy, 1, dummy, ctypes.c_void_p(260), 1 << 20, None) == binding.EWORKSPACE
    assert L.externd_strerror(binding.EHIP).decode().startswith("HIP")


def test_unpack_trits_format():
    # row: [+1, -1, 0, +1, -1] -> codes 01 11 00 01 | 11 (pad 00 00 00)
    b0 = 0b01_00_11_01
    b1 = 0b00_00_00_11
    out = binding.unpack_trits(np.array([[b0, b1]], dtype=np.uint8), 5)
    assert out.tolist() == [[1, -1, 0, 1, -1]]
    with pytest.raises(ValueError):
        binding.unpack_trits(np.array([[0b10, 0]], dtype=np.uint8), 5)       # code 10
    with pytest.raises(ValueError):
        binding.unpack_trits(np.array([[0, 0b0100]], dtype=np.uint8), 5)     # padding bit set


def test_apply_noalloc_rejects_before_device_work():
    """The allocation-free inference entry point checks its arguments and its
    scratch bound on the host: no HIP call is made on these paths."""
    L = binding.lib()
    d = ctypes.c_void_p(256)          # never dereferenced: validation fails first
    f = L.externd_apply_noalloc
    assert f(None, d, d, 10, 10, 10, d, 1, d, None) == binding.EINVAL
    assert f(d, d, d, 10, 10, 10, d, 9, d, None) == binding.EINVAL              # nb above the batch limit
    assert f(d, d, d, 0, 10, 10, d, 1, d, None) == binding.EINVAL
    assert f(d, d, d, 10, 10, 1 << 32, d, 1, d, None) == binding.EUNSUPPORTED
    # the workspace of the call against the fixed bound
    assert binding.APPLY_NOALLOC_MAX_BYTES == 8 << 20
    wsb = L.externd_apply_workspace_bytes
    assert wsb(9728, 2560, 7680, 8) <= binding.APPLY_NOALLOC_MAX_BYTES
    assert wsb(10, 10, 1 << 21, 1) == binding.APPLY_NOALLOC_MAX_BYTES        # exactly fits (4 k bytes)
    assert wsb(10, 10, (1 << 21) + 1, 1) > binding.APPLY_NOALLOC_MAX_BYTES
    assert f(d, d, d, 10, 10, (1 << 21) + 1, d, 1, d, None) == binding.ESCRATCH
    assert wsb(10, 1 << 20, 10, 8) > binding.APPLY_NOALLOC_MAX_BYTES
    assert f(d, d, d, 10, 1 << 20, 10, d, 8, d, None) == binding.ESCRATCH
    assert L.externd_strerror(binding.ESCRATCH).decode().startswith("call exceeds the fixed device scratch")

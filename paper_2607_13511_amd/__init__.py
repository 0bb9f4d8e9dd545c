"""MI355X-native ExTernD factorizer: greedy block-ALS ternary factorization.

A ~= B diag(D) C with B, C in {-1, 0, +1}, computed by hand-written HIP
kernels for gfx950 behind the C-ABI library ``libexternd.so`` (declared in
``include/externd.h``).  ``paper_2607_13511_amd.binding`` is the thin Python
layer over that library; importing this package loads nothing.
"""
__all__ = ["binding", "synth"]

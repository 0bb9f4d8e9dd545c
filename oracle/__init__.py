"""CPU oracle for the ExTernD greedy (block-)ALS ternary factorization.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
link this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library under ``paper_2607_13511_amd/``; the only module both sides use is
the seeded input generator ``paper_2607_13511_amd/synth.py``, which holds none
of the method's arithmetic.
"""
from .externd_oracle import *  # noqa: F401,F403
from .externd_oracle import __all__  # noqa: F401

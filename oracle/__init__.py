"""CPU oracle of the AEP expert-layer hot path -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import, call or execute anything in this package.  The
product (``paper_2505_08944_amd``) never imports it, and it never imports the
product: the two share no code.  Inputs come from ``synth`` (seeded draws
only).

Everything here is the plain, slow definition of the MoE layer that the
paper's asynchronous expert parallelism computes (Sec. 3.2: tokens are queued
per (block, expert) layer, a drained queue is merged into one contiguous batch,
the expert runs, and top-K duplicates are merged back with their gate
weights).  Floating point is evaluated in float64 unless stated otherwise.

Parity status per function is listed in the module docstrings; every function
here is pinned by a ``-m "not gpu"`` test in ``tests/test_oracle_*.py``.
"""

from .moe import *  # noqa: F401,F403
from .scheduler import *  # noqa: F401,F403

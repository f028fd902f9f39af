"""CPU references of the Encode-stage encoder (fp64) and of its micro-batcher
(test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline
leg may import this package; the product path never does.
"""
from . import batcher, encoder  # noqa: F401

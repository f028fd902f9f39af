"""CPU references of the Encode-stage encoder (fp64), its micro-batcher and its
router (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline
leg may import this package; the product path never does.
"""
from . import batcher, encoder, router  # noqa: F401

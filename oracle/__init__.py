"""fp64 CPU reference of the Encode-stage encoder (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s cpu_baseline
leg may import this package; the product path never does.
"""
from . import encoder  # noqa: F401

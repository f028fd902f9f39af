"""Reference of the smallest-safe-share table and its lookup (test
infrastructure only).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py`` may import or call this module; the product path (the binding in
the package) never touches it.

What it computes (paper Section 3.4, dynamic SM partitioning).  Encode latency
is measured at a few SM-allocation levels for a range of batch sizes.  A level's
table entry is the biggest measured batch size that runs at most 20% slower at
that level than on the whole GPU (the threshold drawn in the paper's
latency-versus-allocation figure, the bound itself included).  Given a
micro-batch of B requests, encode takes the smallest level whose entry is at
least B; if no level qualifies, encode keeps the whole GPU (1.0).
"""


def smallest_safe_table(levels, batches, latency, whole_gpu, tolerance=0.2):
    """levels: allocation fractions; batches: batch sizes; latency[level][b] and
    whole_gpu[b]: measured times.  Returns {level: largest safe b, or 0}."""
    table = {}
    for level in levels:
        largest = 0
        for b in batches:
            ok = latency[level][b] <= whole_gpu[b] * (1 + tolerance)
            if ok and b > largest:
                largest = b
        table[level] = largest
    return table


def share_for(table, b):
    """Smallest level whose recorded batch size covers b, else 1.0."""
    for level in sorted(table):
        if table[level] >= b:
            return level
    return 1.0

"""Reference of the deficit-counter router and of the envelope grouping
(test infrastructure only).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py`` may import or call this module; the product path (the C++ router
in the HIP library and its binding) never touches it.

What it computes (paper Section 3.3).  Router: a single real accumulator d,
starting at 0; per request d is increased by the offload ratio s, and the
request's prefill goes to the remote worker when d >= 1 (then d is reduced
by 1), to the local worker otherwise.  The accumulator is an exact rational
here (fractions.Fraction), so the arithmetic is the paper's, not a rounding
of it.  Envelopes: the embeddings of one micro-batch bound for the same
destination are sent as one contiguous block.
"""
from fractions import Fraction


def route(n, s):
    """Decisions (1 = remote) for n requests at offload ratio s (a Fraction
    or anything Fraction accepts)."""
    s = Fraction(s)
    d = Fraction(0)
    out = []
    for _ in range(n):
        d += s
        if d >= 1:
            out.append(1)
            d -= 1
        else:
            out.append(0)
    return out


def envelopes(dest, n_dest, rows):
    """Destination blocks of a micro-batch: for each destination, its requests
    in request order; returns (order, dest_rows, req_rows) with dest_rows the
    n_dest + 1 block offsets and req_rows[i] request i's first row."""
    order, dest_rows, req_rows = [], [0], [None] * len(dest)
    for d in range(n_dest):
        at = dest_rows[-1]
        for i, di in enumerate(dest):
            if di == d:
                order.append(i)
                req_rows[i] = at
                at += rows[i]
        dest_rows.append(at)
    return order, dest_rows, req_rows

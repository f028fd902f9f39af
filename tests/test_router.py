"""Deficit-counter routing and envelope grouping (Section 3.3): the reference
against the paper's worked example and the properties it states, the
library's router and plan against the reference.  Host only."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import router as O
from paper_2609_31551_amd import router as L
from paper_2609_31551_amd.eas import EasError

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "deficit_router_s07.txt")


def _golden():
    f = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        k, *v = line.split()
        f[k] = v
    return Fraction(f["s"][0]), int(f["requests"][0]), [int(x) for x in f["local"]]


def test_reference_reproduces_the_papers_example():
    s, n, local = _golden()
    got = O.route(n, s)
    assert [i + 1 for i, r in enumerate(got) if r == 0] == local
    assert sum(got) == 14                      # about seven remote for every three local


def _runs(seq, v):
    best = cur = 0
    for x in seq:
        cur = cur + 1 if x == v else 0
        best = max(best, cur)
    return best


@pytest.mark.parametrize("s", ["0", "1", "1/2", "7/10", "3/10", "1/3", "9/10", "1/7", "123/1000"])
def test_reference_properties(s):
    """Remote count after every prefix n is floor(n s); runs of remote and
    local decisions stay within ceil(1/(1-s)) and ceil(1/s)."""
    s = Fraction(s)
    seq = O.route(3000, s)
    count = 0
    for n, r in enumerate(seq, 1):
        count += r
        assert count == math.floor(n * s)
    if s < 1:
        assert _runs(seq, 1) <= math.ceil(1 / (1 - s))
    if s > 0:
        assert _runs(seq, 0) <= math.ceil(1 / s)


@pytest.mark.parametrize("s", [0.0, 1.0, 0.5, 0.7, 0.3, 0.123, 0.999999, 0.25])
def test_library_router_matches_reference(s):
    r = L.Router(s)
    assert r.ratio() == s                     # decimal ratios are held exactly
    got = np.concatenate([r.route(k) for k in (1, 7, 0, 500, 1492)])
    ref = O.route(2000, Fraction(str(s)))
    np.testing.assert_array_equal(got, np.array(ref, np.uint8))
    assert r.counts() == (2000, int(sum(ref)))


def test_library_router_example_and_long_run():
    s, n, local = _golden()
    r = L.Router(float(s))
    got = r.route(n)
    assert [i + 1 for i, x in enumerate(got) if x == 0] == local
    r2 = L.Router(0.7)
    r2.route(10 ** 6)
    assert r2.counts() == (10 ** 6, 700000)


def test_router_rejects_bad_ratio():
    for s in (-0.1, 1.5, float("nan")):
        with pytest.raises(EasError):
            L.Router(s)


def test_envelope_plan_matches_reference():
    rng = np.random.default_rng(4)
    for n, nd in ((1, 1), (5, 2), (64, 2), (64, 5), (13, 7)):
        dest = rng.integers(0, nd, n)
        rows = rng.integers(0, 600, n)
        order, dest_rows, req_rows = L.envelope_plan(dest, nd, rows)
        o2, d2, r2 = O.envelopes(list(dest), nd, list(rows))
        assert order.tolist() == o2 and dest_rows.tolist() == d2 and req_rows.tolist() == r2
        # every destination's block is contiguous and in request order
        for d in range(nd):
            members = [i for i in range(n) if dest[i] == d]
            pos = dest_rows[d]
            for i in members:
                assert req_rows[i] == pos
                pos += rows[i]
            assert pos == dest_rows[d + 1]


def test_envelope_plan_rejects_bad_input():
    with pytest.raises(EasError):
        L.envelope_plan([0, 2], 2, [1, 1])
    with pytest.raises(EasError):
        L.envelope_plan([0, 1], 2, [1, -1])

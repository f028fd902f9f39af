"""The smallest-safe-share table and lookup of dynamic SM partitioning
(Section 3.4): the reference pinned to the paper's worked example and to a
latency model with a closed-form answer, the package's implementation checked
against the reference, and the reservation call's host-side argument checks.
No GPU needed."""
import os
import random

import pytest

from oracle import colocate as R

HERE = os.path.dirname(os.path.abspath(__file__))


def _golden():
    table, lookups = {}, []
    levels = sizes = None
    for line in open(os.path.join(HERE, "golden", "sm_partition_example.txt")):
        f = line.split()
        if not f or f[0].startswith("#"):
            continue
        if f[0] == "levels":
            levels = [int(x) / 100 for x in f[1:]]
        elif f[0] == "largest_batch":
            sizes = [int(x) for x in f[1:]]
        elif f[0] == "lookup":
            lookups.append((int(f[1]), int(f[2]) / 100))
    table = dict(zip(levels, sizes))
    return table, lookups


def test_reference_lookup_reproduces_the_papers_example():
    table, lookups = _golden()
    assert len(table) == 5 and lookups
    for b, level in lookups:
        assert R.share_for(table, b) == level
    assert R.share_for(table, 9) == 1.0   # no level sustains 9: the whole GPU


def test_reference_table_on_a_latency_model_with_a_closed_form():
    # latency(level, b) = t(b) * max(1, b / (b0 * level)): the share stops
    # mattering once level >= b / b0; within 20% iff b <= 1.2 * b0 * level
    b0, batches = 10, list(range(1, 65))
    levels = (0.1, 0.3, 0.5, 0.7, 0.9)
    whole = {b: 3.0 + 0.5 * b for b in batches}
    lat = {lv: {b: whole[b] * max(1.0, b / (b0 * lv)) for b in batches} for lv in levels}
    table = R.smallest_safe_table(levels, batches, lat, whole)
    for lv in levels:
        assert table[lv] == min(64, int(1.2 * b0 * lv + 1e-9)), lv
    # exactly 20% slower is still within the threshold; a hair more is not
    lat2 = {0.5: {4: 1.2 * whole[4], 8: 1.2000001 * whole[8]}}
    assert R.smallest_safe_table((0.5,), (4, 8), lat2, whole) == {0.5: 4}
    # nothing within the threshold
    assert R.smallest_safe_table((0.1,), (1, 2), {0.1: {1: 9.0, 2: 9.0}}, whole) == {0.1: 0}


def test_package_table_and_lookup_match_the_reference():
    from paper_2609_31551_amd import colocate as K
    rng = random.Random(3)
    levels, batches = K.LEVELS, (1, 2, 4, 8, 16, 32, 64)
    assert levels == (0.125, 0.3, 0.5, 0.7, 0.9) and K.THRESHOLD == 0.2
    # an unmeasured (stalled) latency never qualifies
    assert K.safe_share_table({0.125: {1: None, 2: 1.0}}, {1: 1.0, 2: 1.0}) == {0.125: 2}
    for _ in range(200):
        whole = {b: rng.uniform(1, 50) for b in batches}
        lat = {lv: {b: whole[b] * rng.uniform(0.95, 3.0) for b in batches} for lv in levels}
        ref = R.smallest_safe_table(levels, batches, lat, whole)
        assert K.safe_share_table(lat, whole) == ref
        for b in (1, 3, 8, 20, 64, 65):
            assert K.select_share(ref, b) == R.share_for(ref, b)
    table, lookups = _golden()
    for b, level in lookups:
        assert K.select_share(table, b) == level


def test_reservation_rejects_bad_arguments_before_any_device_call():
    import ctypes
    from paper_2609_31551_amd import colocate as K
    from paper_2609_31551_amd import eas
    started, release = (ctypes.c_int32 * 4)(), ctypes.c_int32(0)
    p_s, p_r = ctypes.cast(started, ctypes.c_void_p), ctypes.cast(ctypes.pointer(release), ctypes.c_void_p)
    assert K.LIB.eas_cu_reserve(4, 1.0, None, p_r, None) == eas.EAS_ERR_INVALID_ARG
    assert K.LIB.eas_cu_reserve(4, 1.0, p_s, None, None) == eas.EAS_ERR_INVALID_ARG
    assert K.LIB.eas_cu_reserve(4, 0.0, p_s, p_r, None) == eas.EAS_ERR_INVALID_ARG
    assert K.LIB.eas_cu_reserve(4, 61.0, p_s, p_r, None) == eas.EAS_ERR_INVALID_ARG

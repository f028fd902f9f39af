"""Encode saturation-capacity profiling (Section 3.1, Eq. 3) on synthetic
throughput curves with known answers.  Host only."""
import math

import pytest

from paper_2609_31551_amd import capacity as K


def _amdahl(fixed_s, per_item_s):
    # a pass of b items costs fixed + b * per_item: throughput b / (fixed + b per_item)
    return lambda b: b / (fixed_s + b * per_item_s)


def test_doubling_stops_once_a_doubling_gains_under_five_percent():
    f = _amdahl(0.010, 0.0005)      # saturates towards 2000/s
    c_e, b_sat, curve = K.saturation_capacity(f, 1024)
    bs = [b for b, _ in curve]
    assert bs == [2 ** i for i in range(len(bs))]
    gains = [curve[i + 1][1] / curve[i][1] - 1.0 for i in range(len(curve) - 1)]
    assert all(g >= 0.05 for g in gains[:-1]) and gains[-1] < 0.05
    assert c_e == max(v for _, v in curve) and f(b_sat) == c_e
    assert c_e < 2000.0 and c_e > 0.9 * 2000.0


def test_doubling_stops_at_the_largest_batch():
    c_e, b_sat, curve = K.saturation_capacity(lambda b: 100.0 * b, 64)
    assert [b for b, _ in curve] == [1, 2, 4, 8, 16, 32, 64] and b_sat == 64 and c_e == 6400.0


def test_a_throughput_drop_stops_the_doubling_and_keeps_the_best():
    vals = {1: 10.0, 2: 30.0, 4: 50.0, 8: 40.0, 16: 80.0}
    c_e, b_sat, curve = K.saturation_capacity(vals.__getitem__, 16)
    assert [b for b, _ in curve] == [1, 2, 4, 8] and (c_e, b_sat) == (50.0, 4)


def test_utilisation_and_batch_cap():
    assert K.utilization(1200.0, 2, 1000.0) == pytest.approx(0.6)
    assert K.utilization(3000.0, 1, 1500.0) == pytest.approx(2.0)
    assert K.batch_cap(2.0, 1) == 2 and K.batch_cap(7.0, 2) == 4 and K.batch_cap(8.0, 2) == 4
    assert K.batch_cap(0.5, 1) == 1 and math.isclose(K.utilization(0.0, 3, 10.0), 0.0)

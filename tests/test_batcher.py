"""The load-adaptive micro-batcher (Section 3.2, Eq. 5): the reference pinned
against the probability model it is derived from, and the library's C++
batcher against the reference on seeded arrival traces.  Host only."""
import math

import numpy as np
import pytest

from oracle import batcher as O
from paper_2609_31551_amd import batcher as L
from paper_2609_31551_amd import synth
from paper_2609_31551_amd.eas import EasError


# ---- Eq. 5 against what it is defined by ------------------------------------

@pytest.mark.parametrize("B", [2, 3, 8, 32, 64])
@pytest.mark.parametrize("p", [0.1, 0.5, 0.6, 0.9])
def test_kappa_gives_fill_probability_p(B, p):
    """With gaps at most g = kappa / lambda each with probability
    1 - exp(-kappa), all B-1 gaps stay below with probability p."""
    for kappa in (O.kappa(B, p), L.poisson_gap_kappa(B, p)):
        assert abs((1.0 - math.exp(-kappa)) ** (B - 1) - p) < 1e-12


def test_kappa_two_requests_is_exponential_quantile():
    # B = 2: one gap; P(X <= g) = p is the p-quantile of Exp(lambda)
    for p in (0.3, 0.6):
        assert abs(O.kappa(2, p) - (-math.log(1.0 - p))) < 1e-15


def test_threshold_scales_with_inverse_rate_and_grows_with_B():
    g1, g2 = O.gap_threshold(8, 0.6, 10.0), O.gap_threshold(8, 0.6, 40.0)
    assert abs(g1 / g2 - 4.0) < 1e-12
    assert [O.kappa(B, 0.6) < O.kappa(B + 1, 0.6) for B in range(2, 64)] == [True] * 62
    assert O.gap_threshold(1, 0.6, 5.0) == 0.0 == L.poisson_gap_threshold(1, 0.6, 5.0)


def test_threshold_monte_carlo():
    """Exponential gaps at rate lambda: B-1 consecutive gaps all <= g with
    empirical frequency p (200k trials, 4-sigma band)."""
    rng = np.random.default_rng(11)
    B, p, lam = 8, 0.6, 25.0
    g = O.gap_threshold(B, p, lam)
    gaps = rng.exponential(1.0 / lam, size=(200000, B - 1))
    freq = float((gaps.max(axis=1) <= g).mean())
    assert abs(freq - p) < 4 * math.sqrt(p * (1 - p) / 200000)


@pytest.mark.parametrize("B", [4, 16])
def test_batches_fill_with_probability_p_on_poisson_arrivals(B):
    """The whole rule on a Poisson trace with no age cap: a batch fills
    exactly when its B-1 gaps all stay within g, so the fraction of full
    batches approaches p."""
    p, lam = 0.6, 100.0
    arr = synth.arrival_trace(400000, lam, 1.0, seed=5)
    batches = O.dispatch_batches(arr, B, p, lam, max_age=1e9)
    full = sum(len(m) == B for _, m in batches)
    n = len(batches)
    assert abs(full / n - p) < 4 * math.sqrt(p * (1 - p) / n) + 2e-3


# ---- the dispatch rule on hand-worked traces ---------------------------------

def _rate_for_gap(B, p, g):
    return O.kappa(B, p) / g


def test_rule_hand_worked_traces():
    B, p = 3, 0.6
    lam = _rate_for_gap(B, p, 1.0)            # g = 1 s
    assert abs(O.gap_threshold(B, p, lam) - 1.0) < 1e-12
    # fills: the third arrival dispatches at once
    assert [(round(t, 9), m) for t, m in O.dispatch_batches([0.0, 0.5, 0.9], B, p, lam, 10.0)] == \
        [(0.9, [0, 1, 2])]
    # idle gap: nothing for more than g after 0.5 -> leaves at 1.5; the straggler alone at 3.0
    assert [(round(t, 9), m) for t, m in O.dispatch_batches([0.0, 0.5, 2.0], B, p, lam, 10.0)] == \
        [(1.5, [0, 1]), (3.0, [2])]
    # age cap A = 1.2 s: every gap within g, but the batch is cut at 1.2
    assert [(round(t, 9), m) for t, m in O.dispatch_batches([0.0, 0.9, 1.8], 4, p, _rate_for_gap(4, p, 1.0), 1.2)] == \
        [(1.2, [0, 1]), (2.8, [2])]
    # B = 1: each request alone, at its arrival
    assert O.dispatch_batches([0.0, 0.1, 0.1], 1, p, 5.0, 1.0) == [(0.0, [0]), (0.1, [1]), (0.1, [2])]
    assert O.dispatch_batches([], 4, p, 5.0, 1.0) == []


def test_arrival_at_the_deadline_joins():
    B, p = 3, 0.6
    lam = _rate_for_gap(B, p, 0.5)
    g = O.gap_threshold(B, p, lam)
    batches = O.dispatch_batches([0.0, g], B, p, lam, 10.0)
    assert [m for _, m in batches] == [[0, 1]]


# ---- the library's batcher against the reference ----------------------------

def _service(B, per=0.004, fixed=0.006):
    return [0.0] + [fixed + per * s for s in range(1, B + 1)]


@pytest.mark.parametrize("cv", [0.5, 1.0, 2.0])
@pytest.mark.parametrize("B", [1, 8, 64])
@pytest.mark.parametrize("lam", [20.0, 500.0])
def test_library_replay_matches_reference(cv, B, lam):
    arr = synth.arrival_trace(5000, lam, cv, seed=int(cv * 10) + B)
    p, A = 0.6, 1.0
    svc = _service(B)
    got = L.batcher_simulate(arr, B, p, lam, A, svc)
    batches = O.dispatch_batches(list(arr), B, p, lam, A)
    disp, done, size = O.serve(batches, len(arr), svc)
    assert got["n_batches"] == len(batches)
    np.testing.assert_array_equal(got["batch_size"], np.array(size, np.int32))
    np.testing.assert_allclose(got["dispatch_t"], disp, rtol=0, atol=1e-12)
    np.testing.assert_allclose(got["done_t"], done, rtol=0, atol=1e-9)
    assert np.all(got["dispatch_t"] >= arr) and np.all(got["done_t"] > got["dispatch_t"] - 1e-12)


def test_stateful_batcher_reproduces_the_replay():
    """Drive arrive / poll / take with the trace's own clock."""
    B, p, lam, A = 8, 0.6, 200.0, 0.05
    arr = synth.arrival_trace(3000, lam, 1.0, seed=9)
    b = L.Batcher(B, p, lam, A)
    seen = []
    for i, t in enumerate(arr):
        if b.poll(t) and b.deadline() < t:
            seen.append((b.deadline(), b.take()[0]))
        if b.arrive(t, i):
            seen.append((t, b.take()[0]))
    if b.size():
        seen.append((b.deadline(), b.take()[0]))
    ref = O.dispatch_batches(list(arr), B, p, lam, A)
    assert [m for _, m in seen] == [m for _, m in ref]
    assert max(abs(a - c) for (a, _), (c, _) in zip(seen, ref)) < 1e-12


def test_batcher_rejects_bad_use():
    with pytest.raises(EasError):
        L.Batcher(0, 0.6, 1.0)
    with pytest.raises(EasError):
        L.Batcher(8, 1.0, 1.0)
    with pytest.raises(EasError):
        L.poisson_gap_kappa(1, 0.6)
    b = L.Batcher(4, 0.6, 10.0, 1.0)
    assert b.arrive(1.0, 0) is False
    with pytest.raises(EasError):
        b.arrive(0.5, 1)                      # time went backwards
    with pytest.raises(EasError):
        b.arrive(1.0 + b.gap() + 0.01, 1)     # a timeout dispatch was due first
    assert b.size() == 1
    ids, first = b.take()
    assert ids == [0] and first == 1.0 and b.size() == 0 and math.isinf(b.deadline())


def test_gamma_trace_has_the_requested_rate_and_cv():
    for cv in (0.5, 1.0, 2.0):
        g = np.diff(synth.arrival_trace(200000, 40.0, cv, seed=1))
        assert abs(g.mean() * 40.0 - 1.0) < 0.02
        assert abs(g.std() / g.mean() - cv) < 0.03 * cv

"""Reference of the load-adaptive micro-batcher (test infrastructure only).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py`` may import or call this module; the product path (the C++
batcher in the HIP library and its binding) never touches it, and this module
imports nothing from the product package.

What it computes (paper Section 3.2, "Poisson-gap dispatch rule").  The
encode batch bound B is set offline; at run time the batcher decides when a
partial batch leaves.  Arrivals are modelled as Poisson with rate lambda, so
inter-arrival gaps are exponential, P(X <= g) = 1 - exp(-lambda g).  A batch
fills when each of the B-1 gaps after its first request is at most g, with
probability (1 - exp(-lambda g))^(B-1); setting that equal to the target p
gives Eq. 5, kappa = -ln(1 - p^(1/(B-1))) and g = kappa / lambda.  A batch
leaves when it holds B requests, when the idle time since its latest arrival
exceeds g, or when its age since its first arrival exceeds the cap A.

Event semantics used here (the paper states the three conditions; the tie
rule is this reading): a timed-out batch leaves at the first instant a
condition holds, min(latest + g, first + A); an arrival at exactly that
instant still joins, since the conditions are strict inequalities.

The encode worker that consumes the batches is one server working through
them first-in first-out, busy service[s] seconds on a batch of s requests.
"""
import math


def kappa(B, p):
    """Eq. 5: the gap (in mean inter-arrival times) that B-1 consecutive
    exponential gaps all stay below with probability p."""
    if B < 2 or not (0.0 < p < 1.0):
        raise ValueError("kappa needs B >= 2 and 0 < p < 1")
    return -math.log(1.0 - p ** (1.0 / (B - 1)))


def gap_threshold(B, p, lam):
    """g = kappa / lambda (seconds); B = 1 never waits."""
    if lam <= 0:
        raise ValueError("arrival rate must be positive")
    return 0.0 if B == 1 else kappa(B, p) / lam


def dispatch_batches(arrivals, B, p, lam, max_age):
    """Replays the rule over a trace of arrival times (seconds, sorted).

    Returns a list of (dispatch_time, [request indices]) in dispatch order.
    """
    g = gap_threshold(B, p, lam)
    batches = []
    members = []          # the open batch
    first = latest = None
    for i, t in enumerate(arrivals):
        if members:
            leave = min(latest + g, first + max_age)
            if t > leave:                 # idle > g or age > A before this arrival
                batches.append((leave, members))
                members = []
        if not members:
            first = t
        members = members + [i]
        latest = t
        if len(members) == B:             # full: leaves with this arrival
            batches.append((t, members))
            members = []
    if members:
        batches.append((min(latest + g, first + max_age), members))
    return batches


def serve(batches, n_requests, service):
    """One encode server, first in first out: each batch starts when it has
    been dispatched and the previous batch is done.

    Returns per-request lists (dispatch_time, done_time, batch_size)."""
    dispatch = [None] * n_requests
    done = [None] * n_requests
    size = [None] * n_requests
    free = -math.inf
    for t, members in batches:
        start = max(t, free)
        end = start + service[len(members)]
        free = end
        for i in members:
            dispatch[i], done[i], size[i] = t, end, len(members)
    return dispatch, done, size

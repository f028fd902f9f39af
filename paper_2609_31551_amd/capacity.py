"""Encode saturation capacity (paper Section 3.1, Stage 1 of the allocation
search) and the stage utilisation it feeds (Eq. 3).

Encode profiling doubles the micro-batch size B until throughput saturates;
the saturation capacity C_E is the throughput reached.  Reading of
"saturates" (the paper gives no number): the doubling stops once a doubling
raises throughput by less than `min_gain` (5%), or at the largest batch the
worker accepts.  With n_E encode workers sharing a total arrival rate
Lambda, a worker's utilisation is rho_E = (Lambda / n_E) / C_E (Eq. 3), and
the batch bound explored later is capped at ceil(Lambda / n_E).
"""
import math


def saturation_capacity(measure, max_batch, min_gain=0.05):
    """measure(b) -> items per second at micro-batch b.  Returns
    (C_E, b_sat, curve) with curve = [(b, items_per_s), ...] in doubling order;
    C_E is the largest throughput seen and b_sat the batch size reaching it."""
    curve = []
    b = 1
    while b <= max_batch:
        curve.append((b, float(measure(b))))
        if len(curve) >= 2 and curve[-1][1] < (1.0 + min_gain) * curve[-2][1]:
            break
        b *= 2
    b_sat, c_e = max(curve, key=lambda bc: bc[1])
    return c_e, b_sat, curve


def utilization(total_rate, n_workers, capacity):
    """Eq. 3: rho = (Lambda / n) / C."""
    return (total_rate / n_workers) / capacity


def batch_cap(total_rate, n_workers):
    """Largest batch bound worth exploring: ceil(Lambda / n)."""
    return int(math.ceil(total_rate / n_workers))

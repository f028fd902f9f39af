"""ctypes binding of the micro-batcher in libeas.so (include/eas_batcher.h),
same names as the C ABI.  Argument marshalling only; the rule and the trace
replay run in the library's C++."""
import ctypes

import numpy as np

from .eas import LIB, EAS_OK, EasError


class BatcherConfig(ctypes.Structure):
    _fields_ = [("batch_bound", ctypes.c_int32), ("fill_prob", ctypes.c_double),
                ("arrival_rate", ctypes.c_double), ("max_age", ctypes.c_double)]


P, I32, I64, D, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p
_SIG = {
    "eas_poisson_gap_kappa": ([I32, D, P(D)], I32),
    "eas_poisson_gap_threshold": ([I32, D, D, P(D)], I32),
    "eas_batcher_create": ([P(BatcherConfig), P(VP)], I32),
    "eas_batcher_destroy": ([VP], None),
    "eas_batcher_set_rate": ([VP, D], I32),
    "eas_batcher_gap": ([VP, P(D)], I32),
    "eas_batcher_arrive": ([VP, D, I64, P(I32)], I32),
    "eas_batcher_deadline": ([VP, P(D)], I32),
    "eas_batcher_poll": ([VP, D, P(I32)], I32),
    "eas_batcher_take": ([VP, P(I64), I32, P(I32), P(D)], I32),
    "eas_batcher_size": ([VP, P(I32)], I32),
    "eas_batcher_simulate": ([P(BatcherConfig), P(D), I64, P(D), P(D), P(D), P(I32), P(I64)], I32),
}
for _name, (_args, _res) in _SIG.items():
    _fn = getattr(LIB, _name)
    _fn.argtypes = _args
    _fn.restype = _res
EXPORTS = tuple(sorted(_SIG))


def _check(status):
    if status != EAS_OK:
        raise EasError(status)


def _config(B, p, lam, max_age):
    return BatcherConfig(int(B), float(p), float(lam), float(max_age))


def poisson_gap_kappa(B, p):
    k = D()
    _check(LIB.eas_poisson_gap_kappa(int(B), float(p), ctypes.byref(k)))
    return k.value


def poisson_gap_threshold(B, p, lam):
    g = D()
    _check(LIB.eas_poisson_gap_threshold(int(B), float(p), float(lam), ctypes.byref(g)))
    return g.value


class Batcher:
    """Stateful batcher; times are caller-supplied seconds."""

    def __init__(self, B, p, lam, max_age=1.0):
        self.B = int(B)
        self.h = VP()
        self._destroy = LIB.eas_batcher_destroy
        _check(LIB.eas_batcher_create(ctypes.byref(_config(B, p, lam, max_age)), ctypes.byref(self.h)))

    def close(self):
        if self.h:
            self._destroy(self.h)
            self.h = VP()

    def __del__(self):
        self.close()

    def set_rate(self, lam):
        _check(LIB.eas_batcher_set_rate(self.h, float(lam)))

    def gap(self):
        g = D()
        _check(LIB.eas_batcher_gap(self.h, ctypes.byref(g)))
        return g.value

    def arrive(self, t, rid):
        d = I32()
        _check(LIB.eas_batcher_arrive(self.h, float(t), int(rid), ctypes.byref(d)))
        return bool(d.value)

    def deadline(self):
        d = D()
        _check(LIB.eas_batcher_deadline(self.h, ctypes.byref(d)))
        return d.value

    def poll(self, t):
        d = I32()
        _check(LIB.eas_batcher_poll(self.h, float(t), ctypes.byref(d)))
        return bool(d.value)

    def take(self):
        ids = (I64 * self.B)()
        n, first = I32(), D()
        _check(LIB.eas_batcher_take(self.h, ids, self.B, ctypes.byref(n), ctypes.byref(first)))
        return [ids[i] for i in range(n.value)], first.value

    def size(self):
        n = I32()
        _check(LIB.eas_batcher_size(self.h, ctypes.byref(n)))
        return n.value


def batcher_simulate(arrivals, B, p, lam, max_age, service_s):
    """Trace replay of the rule feeding one FIFO encode server.
    service_s[s] = seconds per batch of s requests (index 0 unused)."""
    arr = np.ascontiguousarray(arrivals, dtype=np.float64)
    svc = np.ascontiguousarray(service_s, dtype=np.float64)
    if svc.shape[0] < int(B) + 1:
        raise ValueError("service_s needs batch_bound + 1 entries")
    n = arr.shape[0]
    disp = np.empty(n, np.float64)
    done = np.empty(n, np.float64)
    size = np.empty(n, np.int32)
    nb = I64()
    dp = lambda a: a.ctypes.data_as(P(D))
    _check(LIB.eas_batcher_simulate(ctypes.byref(_config(B, p, lam, max_age)), dp(arr), n, dp(svc), dp(disp),
                                    dp(done), size.ctypes.data_as(P(I32)), ctypes.byref(nb)))
    return {"dispatch_t": disp, "done_t": done, "batch_size": size, "n_batches": nb.value}

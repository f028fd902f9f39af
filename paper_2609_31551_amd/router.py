"""ctypes binding of the deficit-counter router and the envelope calls in
libeas.so (include/eas_router.h), same names as the C ABI.  Argument
marshalling only."""
import ctypes

import numpy as np

from .eas import LIB, EAS_OK, EasError

P, I32, I64, D, VP, U8 = (ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p,
                          ctypes.c_uint8)
_SIG = {
    "eas_router_create": ([D, P(VP)], I32),
    "eas_router_destroy": ([VP], None),
    "eas_router_ratio": ([VP, P(D)], I32),
    "eas_router_route": ([VP, I64, P(U8)], I32),
    "eas_router_counts": ([VP, P(I64), P(I64)], I32),
    "eas_envelope_plan": ([I32, P(I32), I32, P(I64), P(I32), P(I64), P(I64)], I32),
    "eas_envelope_gather": ([VP, P(I64), P(I64), I32, I64, VP, VP], I32),
}
for _name, (_args, _res) in _SIG.items():
    _fn = getattr(LIB, _name)
    _fn.argtypes = _args
    _fn.restype = _res
EXPORTS = tuple(sorted(_SIG))


def _check(status):
    if status != EAS_OK:
        raise EasError(status)


class Router:
    def __init__(self, offload_ratio):
        self.h = VP()
        self._destroy = LIB.eas_router_destroy
        _check(LIB.eas_router_create(float(offload_ratio), ctypes.byref(self.h)))

    def close(self):
        if self.h:
            self._destroy(self.h)
            self.h = VP()

    def __del__(self):
        self.close()

    def ratio(self):
        s = D()
        _check(LIB.eas_router_ratio(self.h, ctypes.byref(s)))
        return s.value

    def route(self, n):
        out = np.empty(int(n), np.uint8)
        _check(LIB.eas_router_route(self.h, int(n), out.ctypes.data_as(P(U8))))
        return out

    def counts(self):
        routed, remote = I64(), I64()
        _check(LIB.eas_router_counts(self.h, ctypes.byref(routed), ctypes.byref(remote)))
        return routed.value, remote.value


def envelope_plan(dest, n_dest, rows):
    dest = np.ascontiguousarray(dest, np.int32)
    rows = np.ascontiguousarray(rows, np.int64)
    n = dest.shape[0]
    order = np.empty(n, np.int32)
    dest_rows = np.empty(int(n_dest) + 1, np.int64)
    req_rows = np.empty(n, np.int64)
    _check(LIB.eas_envelope_plan(n, dest.ctypes.data_as(P(I32)), int(n_dest), rows.ctypes.data_as(P(I64)),
                                 order.ctypes.data_as(P(I32)), dest_rows.ctypes.data_as(P(I64)),
                                 req_rows.ctypes.data_as(P(I64))))
    return order, dest_rows, req_rows


def envelope_gather(src, src_rows, req_rows, dst, stream=None):
    """src, dst: device tensors [rows, dim]; src_rows (n + 1) and req_rows (n)
    host arrays.  Enqueued on `stream` (torch stream or None)."""
    import torch
    src_rows = np.ascontiguousarray(src_rows, np.int64)
    req_rows = np.ascontiguousarray(req_rows, np.int64)
    row_bytes = src.shape[1] * src.element_size()
    s = (stream or torch.cuda.current_stream()).cuda_stream
    _check(LIB.eas_envelope_gather(ctypes.c_void_p(src.data_ptr()), src_rows.ctypes.data_as(P(I64)),
                                   req_rows.ctypes.data_as(P(I64)), req_rows.shape[0], row_bytes,
                                   ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(s)))

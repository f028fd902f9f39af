"""ctypes binding of libeas.so (include/eas_encoder.h), same names as the C ABI.

Argument marshalling only: every step of the Encode path runs in the HIP
library.  PyTorch supplies device memory and the stream.  Importing this
module loads the library and raises if it has not been built.
"""
import ctypes
import os

import numpy as np
import torch

from . import configs as C

_HERE = os.path.dirname(os.path.abspath(__file__))
# EAS_LIBRARY names another build of the same sources (the host-sanitized test
# build); by default the in-tree library
LIB_PATH = os.environ.get("EAS_LIBRARY") or os.path.join(_HERE, "libeas.so")

EAS_OK, EAS_ERR_INVALID_ARG, EAS_ERR_SHAPE, EAS_ERR_CAPACITY, EAS_ERR_UNSUPPORTED, EAS_ERR_HIP = range(6)
EAS_MAX_SEQS = 64
_KIND = {C.KIND_VIT_ABS: 0, C.KIND_VIT_CLS_ABS: 1, C.KIND_VIT_ROPE: 2, C.KIND_WHISPER: 3}
_DTYPE = {"fp32": 0, "bf16": 1}
_ACT = {"gelu": 0, "quick_gelu": 1}


class Config(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("dtype", ctypes.c_int32), ("layers", ctypes.c_int32),
                ("hidden", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("mlp", ctypes.c_int32), ("act", ctypes.c_int32), ("in_chans", ctypes.c_int32),
                ("patch", ctypes.c_int32), ("temporal_patch", ctypes.c_int32), ("merge", ctypes.c_int32),
                ("out_dim", ctypes.c_int32), ("ln_eps", ctypes.c_float), ("merger_ln_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_float), ("rope_sections", ctypes.c_int32 * 3),
                ("pos_grid", ctypes.c_int32 * 2), ("n_mels", ctypes.c_int32), ("n_frames", ctypes.c_int32),
                ("max_tokens", ctypes.c_int64), ("max_seqs", ctypes.c_int32), ("out_dtype", ctypes.c_int32)]


class TensorDesc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 48), ("offset_bytes", ctypes.c_int64), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 2)]


class KernelStat(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_char * 64), ("launches", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("flops", ctypes.c_double), ("bytes", ctypes.c_double)]


EXPORTS = ("eas_encoder_create", "eas_encoder_destroy", "eas_weights_layout", "eas_microbatch_shape",
           "eas_validate_microbatch", "eas_pack_microbatch", "eas_encode_microbatch", "eas_profile_enable",
           "eas_profile_read", "eas_status_string", "eas_last_error", "eas_encode_microbatch_noalloc",
           "eas_mfma_rate_probe")
EAS_NOALLOC_SCRATCH_BYTES = 256 << 20


def _load():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libeas.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, I64, VP = ctypes.POINTER, ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p
    sig = {
        "eas_encoder_create": ([P(Config), P(VP)], I32),
        "eas_encoder_destroy": ([VP], None),
        "eas_weights_layout": ([P(Config), P(TensorDesc), I32, P(I32), P(I64)], I32),
        "eas_microbatch_shape": ([P(Config), I32, P(I32), P(I32), P(I32), P(I64), P(I64)], I32),
        "eas_validate_microbatch": ([P(Config), P(I32), P(I32), I32], I32),
        "eas_pack_microbatch": ([VP, I32, P(VP), P(I32), VP, P(I32), P(I32), VP], I32),
        "eas_encode_microbatch": ([VP, VP, P(I32), P(I32), I32, VP, VP, P(I32), VP], I32),
        "eas_profile_enable": ([VP, I32], I32),
        "eas_profile_read": ([VP, P(KernelStat), I32, P(I32)], I32),
        "eas_status_string": ([I32], ctypes.c_char_p),
        "eas_last_error": ([VP], ctypes.c_char_p),
        "eas_encode_microbatch_noalloc": ([P(Config), VP, P(I32), P(I32), I32, VP, VP, P(I32), VP], I32),
        "eas_mfma_rate_probe": ([I32, I32, P(ctypes.c_double), VP], I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


LIB = _load()


class EasError(RuntimeError):
    def __init__(self, status, detail=""):
        self.status = status
        msg = LIB.eas_status_string(status).decode()
        super().__init__("%s (%d)%s" % (msg, status, (": " + detail) if detail else ""))


def _check(status, handle=None):
    if status != EAS_OK:
        detail = LIB.eas_last_error(handle).decode() if handle else ""
        raise EasError(status, detail)


def make_config(preset, max_tokens=1, max_seqs=EAS_MAX_SEQS, out_dtype="fp32"):
    c = Config()
    c.kind = _KIND[preset["kind"]]
    c.dtype = _DTYPE[preset["dtype"]]
    c.act = _ACT[preset["act"]]
    for f in ("layers", "hidden", "heads", "head_dim", "mlp", "in_chans", "patch", "temporal_patch", "merge",
              "out_dim", "n_mels", "n_frames"):
        setattr(c, f, int(preset[f]))
    c.ln_eps, c.merger_ln_eps, c.rope_theta = preset["ln_eps"], preset["merger_ln_eps"], preset["rope_theta"]
    for i in range(3):
        c.rope_sections[i] = int(preset["rope_sections"][i])
    for i in range(2):
        c.pos_grid[i] = int(preset["pos_grid"][i])
    c.max_tokens, c.max_seqs, c.out_dtype = int(max_tokens), int(max_seqs), _DTYPE[out_dtype]
    return c


def _i32(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def weights_layout(cfg):
    """[(name, offset_bytes, shape)], total_bytes"""
    n = ctypes.c_int32()
    total = ctypes.c_int64()
    _check(LIB.eas_weights_layout(ctypes.byref(cfg), None, 0, ctypes.byref(n), ctypes.byref(total)))
    descs = (TensorDesc * n.value)()
    _check(LIB.eas_weights_layout(ctypes.byref(cfg), descs, n.value, ctypes.byref(n), ctypes.byref(total)))
    out = [(d.name.decode(), d.offset_bytes, tuple(d.shape[i] for i in range(d.ndim))) for d in descs]
    return out, total.value


def microbatch_shape(cfg, tchw):
    tchw, p = _i32(tchw)
    n = tchw.shape[0]
    cu, pcu = _i32(np.zeros(n + 1))
    grid, pg = _i32(np.zeros((n, 3)))
    pe, orow = ctypes.c_int64(), ctypes.c_int64()
    _check(LIB.eas_microbatch_shape(ctypes.byref(cfg), n, p, pcu, pg, ctypes.byref(pe), ctypes.byref(orow)))
    return cu, grid, pe.value, orow.value


def validate_microbatch(cfg, cu_seqlens, grid_thw, n_seqs=None):
    """Returns the eas_status (host-only check)."""
    cu, pcu = _i32(cu_seqlens)
    pg = None
    if grid_thw is not None:
        grid, pg = _i32(grid_thw)
    n = len(cu) - 1 if n_seqs is None else n_seqs
    return LIB.eas_validate_microbatch(ctypes.byref(cfg), pcu, pg, n)


def _to_bf16_bits(a):
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)).astype(np.uint16)


def upload_weights(cfg, weights, device="cuda"):
    """Place a dict name -> array into one flat device buffer in the library's
    canonical layout (rounded to the model dtype)."""
    layout, total = weights_layout(cfg)
    host = np.zeros(total, dtype=np.uint8)
    bf16 = cfg.dtype == _DTYPE["bf16"]
    for name, off, shape in layout:
        a = np.asarray(weights[name], dtype=np.float32)
        if tuple(a.shape) != tuple(shape):
            raise ValueError("weight %s has shape %s, layout wants %s" % (name, a.shape, shape))
        raw = (_to_bf16_bits(a) if bf16 else a).reshape(-1).view(np.uint8)
        host[off:off + raw.size] = raw
    return torch.from_numpy(host).to(device)


def _stream_ptr(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def mfma_rate_probe(zero_operands=False, iters=50000, stream=None):
    """Dense bf16 TFLOP/s of back-to-back MFMAs on register-resident random (or
    all-zero) operands on every CU (eas_mfma_rate_probe; measurement only)."""
    t = ctypes.c_double()
    _check(LIB.eas_mfma_rate_probe(1 if zero_operands else 0, int(iters), ctypes.byref(t), _stream_ptr(stream)))
    return t.value


def encode_microbatch_noalloc(cfg, packed, cu_seqlens, grid_thw, weights, out, stream=None):
    """eas_encode_microbatch_noalloc: the Encode pass with no handle and no
    allocation (workspace in the library's fixed per-device array).  ``out``
    is the caller's [rows, out_dim] tensor.  Returns cu_out."""
    cu, pcu = _i32(cu_seqlens)
    pg = None
    if grid_thw is not None:
        g, pg = _i32(grid_thw)
    n = len(cu) - 1
    cu_out, pco = _i32(np.zeros(n + 1))
    _check(LIB.eas_encode_microbatch_noalloc(ctypes.byref(cfg), ctypes.c_void_p(packed.data_ptr()), pcu, pg, n,
                                             ctypes.c_void_p(weights.data_ptr()), ctypes.c_void_p(out.data_ptr()),
                                             pco, _stream_ptr(stream)))
    return cu_out


class Encoder:
    """One eas_encoder handle (workspace for max_tokens tokens, max_seqs requests)."""

    def __init__(self, preset, max_tokens, max_seqs=EAS_MAX_SEQS, out_dtype="fp32"):
        self.preset = preset
        self.cfg = make_config(preset, max_tokens, max_seqs, out_dtype)
        self.torch_dtype = torch.bfloat16 if preset["dtype"] == "bf16" else torch.float32
        self.out_torch_dtype = torch.bfloat16 if out_dtype == "bf16" else torch.float32
        h = ctypes.c_void_p()
        _check(LIB.eas_encoder_create(ctypes.byref(self.cfg), ctypes.byref(h)))
        self.h = h

    def close(self):
        if self.h:
            LIB.eas_encoder_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def pack_microbatch(self, items, stream=None):
        """items: list of fp32 CUDA tensors ([frames, C, H, W] or [n_mels, n_frames]).
        Returns (packed, cu_seqlens, grid_thw)."""
        n = len(items)
        tchw = np.array([list(t.shape) if t.dim() == 4 else [1, 1] + list(t.shape) for t in items], np.int32)
        cu, grid, elems, _ = microbatch_shape(self.cfg, tchw)
        packed = torch.empty(elems, dtype=self.torch_dtype, device=items[0].device)
        ptrs = (ctypes.c_void_p * n)(*[t.data_ptr() for t in items])
        for t in items:
            if t.dtype != torch.float32 or not t.is_contiguous() or not t.is_cuda:
                raise ValueError("items must be contiguous fp32 CUDA tensors")
        _, ptch = _i32(tchw)
        cu_o, pcu = _i32(np.zeros(n + 1))
        grid_o, pg = _i32(np.zeros((n, 3)))
        _check(LIB.eas_pack_microbatch(self.h, n, ptrs, ptch, ctypes.c_void_p(packed.data_ptr()), pcu, pg,
                                       _stream_ptr(stream)), self.h)
        return packed, cu_o, grid_o

    def out_rows(self, cu_seqlens):
        n = int(cu_seqlens[-1])
        return n // 4 if self.preset["merge"] == 2 else n

    def encode_microbatch(self, packed, cu_seqlens, grid_thw, weights, out=None, stream=None):
        """Returns (out_embeddings [rows, out_dim], cu_out)."""
        cu, pcu = _i32(cu_seqlens)
        pg = None
        if grid_thw is not None:
            g, pg = _i32(grid_thw)
        n = len(cu) - 1
        if out is None:
            out = torch.empty((self.out_rows(cu), self.preset["out_dim"]), dtype=self.out_torch_dtype,
                              device=packed.device)
        if packed.dtype != self.torch_dtype:
            raise ValueError("packed input must be %s" % self.torch_dtype)
        cu_out, pco = _i32(np.zeros(n + 1))
        _check(LIB.eas_encode_microbatch(self.h, ctypes.c_void_p(packed.data_ptr()), pcu, pg, n,
                                         ctypes.c_void_p(weights.data_ptr()), ctypes.c_void_p(out.data_ptr()), pco,
                                         _stream_ptr(stream)), self.h)
        return out, cu_out

    def profile_enable(self, on=True):
        _check(LIB.eas_profile_enable(self.h, 1 if on else 0), self.h)

    def profile_read(self):
        n = ctypes.c_int32()
        _check(LIB.eas_profile_read(self.h, None, 0, ctypes.byref(n)), self.h)
        stats = (KernelStat * max(1, n.value))()
        _check(LIB.eas_profile_read(self.h, stats, n.value, ctypes.byref(n)), self.h)
        return {s.kernel.decode(): dict(launches=s.launches, ms=s.total_ms, flops=s.flops, bytes=s.bytes)
                for s in stats[:n.value]}

"""Host-side checks of the C ABI: the library loads, exports every symbol the
header declares, lays weights out in the canonical order, and rejects bad
micro-batches before any device work.  No GPU needed (no HIP compute call)."""
import os
import re

import numpy as np
import pytest

from paper_2609_31551_amd import configs as C
from paper_2609_31551_amd import eas
from paper_2609_31551_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "eas_encoder.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:eas_status|void|const char\*)\s+(eas_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(eas.LIB, n), n
    assert sorted(eas.EXPORTS) == names


def test_every_batcher_symbol_is_exported():
    from paper_2609_31551_amd import batcher
    text = open(os.path.join(ROOT, "include", "eas_batcher.h")).read()
    names = sorted(set(re.findall(r"^\s*(?:eas_status|void)\s+(eas_\w+)\s*\(", text, re.M)))
    assert len(names) == 12
    for n in names:
        assert hasattr(eas.LIB, n), n
    assert list(batcher.EXPORTS) == names


@pytest.mark.parametrize("preset", list(C.PRESETS.values()), ids=list(C.PRESETS))
def test_weight_layout_matches_generator_tensor_list(preset):
    cfg = eas.make_config(C.with_layers(preset, 2), max_tokens=1024)
    layout, total = eas.weights_layout(cfg)
    specs = synth.weight_specs(C.with_layers(preset, 2))
    assert [n for n, _, _ in layout] == [n for n, _, _ in specs]
    assert [tuple(s) for _, _, s in layout] == [tuple(s) for _, s, _ in specs]
    el = 2 if preset["dtype"] == "bf16" else 4
    offs = [o for _, o, _ in layout]
    assert offs[0] == 0 and all(o % 256 == 0 for o in offs)
    for (n, o, s), o2 in zip(layout, offs[1:] + [total]):
        assert o + int(np.prod(s)) * el <= o2


def test_microbatch_shape_counts_tokens_and_cls():
    cfg = eas.make_config(C.CLIP_L336, max_tokens=4096, max_seqs=8)
    cu, grid, elems, rows = eas.microbatch_shape(cfg, [[1, 3, 336, 336]] * 3)
    assert cu.tolist() == [0, 577, 1154, 1731]
    assert grid.tolist() == [[1, 24, 24]] * 3
    assert elems == 1731 * 588 and rows == 1731
    cfg = eas.make_config(C.QWEN_IMAGE, max_tokens=100000, max_seqs=8)
    cu, grid, elems, rows = eas.microbatch_shape(cfg, [[2, 3, 224, 308], [2, 3, 1344, 672]])
    assert cu.tolist() == [0, 16 * 22, 16 * 22 + 96 * 48]
    assert grid.tolist() == [[1, 16, 22], [1, 96, 48]]
    assert rows == cu[-1] // 4 and elems == cu[-1] * 1176
    cfg = eas.make_config(C.WHISPER_L, max_tokens=10000, max_seqs=8)
    cu, _, elems, rows = eas.microbatch_shape(cfg, [[1, 1, 128, 3000]] * 2)
    assert cu.tolist() == [0, 1500, 3000] and elems == 2 * 128 * 3000 and rows == 3000


def test_validate_accepts_good_and_rejects_bad_batches():
    cfg = eas.make_config(C.QWEN_IMAGE, max_tokens=2000, max_seqs=4)
    good_grid = [[1, 16, 22], [1, 8, 8]]
    assert eas.validate_microbatch(cfg, [0, 352, 416], good_grid) == eas.EAS_OK
    assert eas.validate_microbatch(cfg, [1, 352, 416], good_grid) == eas.EAS_ERR_SHAPE          # cu[0] != 0
    assert eas.validate_microbatch(cfg, [0, 352, 352], good_grid) == eas.EAS_ERR_SHAPE          # not increasing
    assert eas.validate_microbatch(cfg, [0, 350, 414], good_grid) == eas.EAS_ERR_SHAPE          # grid mismatch
    assert eas.validate_microbatch(cfg, [0, 15 * 22, 15 * 22 + 64], [[1, 15, 22], [1, 8, 8]]) == eas.EAS_ERR_SHAPE  # odd h
    assert eas.validate_microbatch(cfg, [0, 2112], [[1, 48, 44]]) == eas.EAS_ERR_CAPACITY     # > max_tokens
    assert eas.validate_microbatch(cfg, [0] + [64] * 5, [[1, 8, 8]] * 5, 5) == eas.EAS_ERR_CAPACITY  # > max_seqs
    assert eas.validate_microbatch(cfg, [0, 352], None) == eas.EAS_ERR_INVALID_ARG            # grid required
    cfgc = eas.make_config(C.CLIP_L336, max_tokens=4096, max_seqs=4)
    assert eas.validate_microbatch(cfgc, [0, 577], [[1, 24, 24]]) == eas.EAS_OK
    assert eas.validate_microbatch(cfgc, [0, 576], [[1, 24, 24]]) == eas.EAS_ERR_SHAPE        # CLS token missing
    assert eas.validate_microbatch(cfgc, [0, 626], [[1, 25, 25]]) == eas.EAS_ERR_SHAPE        # beyond the pos table
    cfgw = eas.make_config(C.WHISPER_L, max_tokens=4096, max_seqs=4)
    assert eas.validate_microbatch(cfgw, [0, 1500, 3000], None) == eas.EAS_OK
    assert eas.validate_microbatch(cfgw, [0, 1500, 2999], None) == eas.EAS_ERR_SHAPE


def test_config_errors_are_reported_without_hip():
    bad = dict(C.CLIP_L336, heads=15)
    cfg = eas.make_config(bad, max_tokens=10)
    assert eas.validate_microbatch(cfg, [0, 577], [[1, 24, 24]]) == eas.EAS_ERR_INVALID_ARG
    odd = dict(C.QWEN_IMAGE, head_dim=40, heads=32, rope_sections=(0, 10, 10))
    cfg = eas.make_config(odd, max_tokens=10)
    assert eas.validate_microbatch(cfg, [0, 4], [[1, 2, 2]]) == eas.EAS_ERR_UNSUPPORTED
    with pytest.raises(eas.EasError):
        eas.weights_layout(eas.make_config(dict(C.QWEN_IMAGE, rope_sections=(0, 20, 19)), max_tokens=10))
    with pytest.raises(eas.EasError):
        eas.microbatch_shape(eas.make_config(C.QWEN_IMAGE, max_tokens=10 ** 5), [[2, 3, 230, 308]])


def test_mfma_probe_rejects_bad_arguments_without_hip():
    import ctypes
    t = ctypes.c_double()
    assert eas.LIB.eas_mfma_rate_probe(0, 0, ctypes.byref(t), None) == eas.EAS_ERR_INVALID_ARG
    assert eas.LIB.eas_mfma_rate_probe(0, (1 << 20) + 1, ctypes.byref(t), None) == eas.EAS_ERR_INVALID_ARG
    assert eas.LIB.eas_mfma_rate_probe(0, 100, None, None) == eas.EAS_ERR_INVALID_ARG


@pytest.mark.parametrize("preset", [C.CLIP_L336, C.QWEN_IMAGE, C.WHISPER_L, C.TINY], ids=lambda p: p["name"])
def test_max_tokens_is_capped_where_32_bit_offsets_end(preset):
    """A handle's widest per-token buffer (MLP hidden, qkv, merger input,
    padded patch rows) stays below 2^31 elements, so every bf16 kernel's
    32-bit byte offsets hold and no micro-batch size changes the kernel (and
    so the bits) a request gets.  Refused with UNSUPPORTED beyond that, on the
    host, before any HIP call."""
    d, f = preset["hidden"], preset["mlp"]
    widest = max(3 * d, f, 4 * d, (C.k_patch(preset) + 63) // 64 * 64)
    if preset["kind"] == C.KIND_WHISPER:
        widest = max(widest, 6 * preset["n_mels"])
    limit = (2 ** 31 - 1) // widest      # largest accepted max_tokens
    ok = eas.make_config(preset, max_tokens=limit, max_seqs=2)
    assert eas.weights_layout(ok)[1] > 0
    for mt in (limit + 1, 2 ** 30):
        cfg = eas.make_config(preset, max_tokens=mt, max_seqs=2)
        assert eas.validate_microbatch(cfg, [0, 4], [[1, 2, 2]]) == eas.EAS_ERR_UNSUPPORTED
    if preset is C.QWEN_IMAGE:
        assert limit == 419430             # 32 of the largest images (9216 tokens) fit


def test_every_router_symbol_is_exported():
    from paper_2609_31551_amd import router
    text = open(os.path.join(ROOT, "include", "eas_router.h")).read()
    names = sorted(set(re.findall(r"^\s*(?:eas_status|void)\s+(eas_\w+)\s*\(", text, re.M)))
    assert len(names) == 7
    for n in names:
        assert hasattr(eas.LIB, n), n
    assert list(router.EXPORTS) == names


def test_every_colocation_symbol_is_exported():
    from paper_2609_31551_amd import colocate
    text = open(os.path.join(ROOT, "include", "eas_colocate.h")).read()
    names = sorted(set(re.findall(r"^\s*(?:eas_status|void|int32_t)\s+(eas_\w+)\s*\(", text, re.M)))
    assert names == ["eas_cu_reserve", "eas_cu_reserve_max"]
    for n in names:
        assert hasattr(eas.LIB, n), n
    assert list(colocate.EXPORTS) == names


def test_cu_reservation_keeps_one_cu_per_shader_engine_free():
    """gfx950 has shader engines of 8 CUs: a reservation may take all but one
    CU of each (224 of MI355X's 256), and larger shares are refused."""
    from paper_2609_31551_amd import colocate
    assert colocate.reserve_max(256) == 224
    assert colocate.reserve_max(304) == 266
    assert colocate.reserve_max(8) == 7 and colocate.reserve_max(1) == 0 and colocate.reserve_max(0) == 0
    assert colocate.reserve_max(-5) == 0
    # the profile's smallest encode share (12.5%) reserves exactly the limit
    assert 256 - round(colocate.LEVELS[0] * 256) == colocate.reserve_max(256)

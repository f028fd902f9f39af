"""The bf16 storage model (tests/_storage_model.py) against the reference.

Pins: with rounding off it is the reference's forward pass for every encoder
kind.  Then the reading it supports: on the nearly one-hot attention workload
(q / k weights of std 0.2) bf16 storage alone moves a Qwen-style encoder's
embeddings by more than 1.5% of max|ref| from the exact result, most of the
2e-2 bf16 bar, while on ordinary weights it costs well under 1%.
"""
import numpy as np
import pytest

import _storage_model as storage_model
from _harness import peaked_weights, rel_err
from oracle import encoder as O
from paper_2609_31551_amd import configs as C
from paper_2609_31551_amd import synth
from test_oracle_pins import rand_weights, small_cfg


def _small_items(cfg, rng):
    if cfg["kind"] == C.KIND_WHISPER:
        return [rng.normal(size=(cfg["n_mels"], cfg["n_frames"])) for _ in range(2)]
    shapes = {C.KIND_VIT_ABS: [(1, 16, 8), (1, 8, 8)], C.KIND_VIT_CLS_ABS: [(1, 12, 12), (1, 8, 12)],
              C.KIND_VIT_ROPE: [(2, 16, 8), (4, 8, 8)]}[cfg["kind"]]
    return [rng.random((t, cfg["in_chans"], h, w)) for t, h, w in shapes]


@pytest.mark.parametrize("kind", [C.KIND_VIT_ABS, C.KIND_VIT_CLS_ABS, C.KIND_VIT_ROPE, C.KIND_WHISPER])
def test_without_rounding_it_is_the_reference(kind):
    cfg = small_cfg(kind)
    rng = np.random.default_rng(5)
    W = rand_weights(cfg, 6)
    items = _small_items(cfg, rng)
    packed, cu, grid = O.pack(cfg, items)
    ref, ref_cu = O.encode(cfg, W, packed, cu, grid)
    got, got_cu = storage_model.encode(cfg, W, packed, cu, grid, rounding=False)
    np.testing.assert_array_equal(got_cu, ref_cu)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12 * np.abs(ref).max())
    rounded, _ = storage_model.encode(cfg, W, packed, cu, grid)
    assert 0.0 < rel_err(rounded, ref) < 2e-2


def test_bf16_storage_alone_costs_most_of_the_bar_on_nearly_one_hot_rows():
    p = C.with_layers(C.QWEN_IMAGE, 1)
    items = synth.make_items(p, 2, 0, shapes=[(2, 224, 308), (2, 392, 224)])
    packed, cu, grid = O.pack(p, items)
    errs = {}
    for std in (None, 0.2):
        W = peaked_weights(p, 3, qk_std=std)
        ref, _ = O.encode(p, W, packed, cu, grid)
        stored, _ = storage_model.encode(p, W, packed, cu, grid)
        errs[std] = rel_err(stored, ref)
    print("bf16 storage vs exact: logit std ~4: %.3g, nearly one-hot: %.3g" % (errs[None], errs[0.2]))
    assert errs[None] < 6e-3
    assert errs[0.2] > 1.5e-2

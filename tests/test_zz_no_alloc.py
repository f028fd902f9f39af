"""The allocation-free entry point (eas_encode_microbatch_noalloc) against the
handle-based one (eas_encode_microbatch), through the C ABI.

For each encoder kind two calls in a row on the library's fixed scratch
array -- a micro-batch, then a smaller one -- must give bit-identical
embeddings and the same cu_out as the handle-based entry point on the same
inputs.  The refusal of a micro-batch beyond the array is a host-side check.
"""
import numpy as np
import pytest
import torch

from paper_2609_31551_amd import configs as C
from paper_2609_31551_amd import eas, synth

CASES = {
    "clip_vit_l14_336": (C.with_layers(C.CLIP_L336, 2), None, (3, 1)),
    "qwen2vl_vit_image": (C.with_layers(C.QWEN_IMAGE, 2), [(2, 224, 308), (2, 392, 224), (2, 280, 280)], (3, 1)),
    "qwen2vl_vit_video": (C.with_layers(C.QWEN_VIDEO, 2), [(4, 112, 168), (6, 56, 112)], (2, 1)),
    "whisper_large_enc": (C.with_layers(C.WHISPER_L, 2), None, (2, 1)),
}


def _run_both(p, items, W):
    n = len(items)
    enc = eas.Encoder(p, max_tokens=1 << 16, max_seqs=n)
    wdev = eas.upload_weights(enc.cfg, W)
    packed, cu, grid = enc.pack_microbatch([torch.from_numpy(a).cuda() for a in items])
    g = None if p["kind"] == C.KIND_WHISPER else grid
    ref, ref_cu = enc.encode_microbatch(packed, cu, g, wdev)
    out = torch.full_like(ref, float("nan"))
    got_cu = eas.encode_microbatch_noalloc(enc.cfg, packed, cu, g, wdev, out)
    torch.cuda.synchronize()
    enc.close()
    return ref.cpu().numpy(), ref_cu, out.cpu().numpy(), got_cu


@pytest.mark.gpu
@pytest.mark.parametrize("name", list(CASES))
def test_noalloc_matches_handle_entry_point_on_two_calls(name):
    p, shapes, (n1, n2) = CASES[name]
    W = synth.make_weights(p, 0)
    all_items = synth.make_items(p, n1, 0, shapes=shapes)
    for n in (n1, n2):   # the second call is smaller and reuses the array the first one left behind
        ref, ref_cu, got, got_cu = _run_both(p, all_items[:n], W)
        print("[noalloc] %s: %d requests, %d output rows" % (p["name"], n, ref.shape[0]), flush=True)
        np.testing.assert_array_equal(got_cu, ref_cu)
        np.testing.assert_array_equal(got, ref)


def test_noalloc_refuses_micro_batches_beyond_its_array():
    """Host-side: a CLIP micro-batch of 25 images (14425 tokens) needs more
    than the fixed array holds and is refused with CAPACITY before any HIP
    call (no device pointer is touched, so fake ones do)."""
    p = C.CLIP_L336
    cfg = eas.make_config(p, max_tokens=1 << 16, max_seqs=64)
    fake = torch.empty(1)
    for n, want in ((25, eas.EAS_ERR_CAPACITY),):
        cu = np.arange(n + 1) * 577
        grid = np.tile([1, 24, 24], (n, 1))
        with pytest.raises(eas.EasError) as e:
            eas.encode_microbatch_noalloc(cfg, fake, cu, grid, fake, fake, stream=_FakeStream())
        assert e.value.status == want


class _FakeStream:
    cuda_stream = 0

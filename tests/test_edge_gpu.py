"""GPU edge cases: the smallest requests the method admits, and calls the
library must refuse.

* Degenerate sizes: a 28 x 28 image (a 2 x 2 patch grid, 4 tokens, one merger
  window, attention over 4 keys) and a one-frame-pair 28 x 28 clip, micro-batched
  with ordinary requests; each must match the fp64 reference and be
  bit-identical to its own micro-batch-1 encoding.
* Refused calls: an empty micro-batch, more requests than max_seqs, more tokens
  than max_tokens and a cu_seqlens / grid_thw mismatch are rejected on the host
  (the documented status, nothing written to the output), and the handle then
  encodes a valid micro-batch exactly as before.
"""
import numpy as np
import pytest

from _harness import check_parity, gpu_encode, oracle_encode
from paper_2609_31551_amd import configs as C
from paper_2609_31551_amd import synth

pytestmark = pytest.mark.gpu

CASES = {
    "qwen_image": (C.QWEN_IMAGE, [(2, 28, 28), (2, 56, 28), (2, 280, 308), (2, 28, 28)]),   # 4, 8, 440, 4 tokens
    "qwen_video": (C.QWEN_VIDEO, [(2, 28, 28), (4, 56, 56), (2, 28, 28)]),                  # 4, 32, 4 tokens
}


@pytest.mark.parametrize("case", list(CASES))
def test_smallest_requests_match_reference_and_single_calls(case):
    base, shapes = CASES[case]
    p = C.with_layers(base, 2)
    W = synth.make_weights(p, 0)
    items = synth.make_items(p, len(shapes), 0, shapes=shapes)
    got = gpu_encode(p, items, W)
    check_parity(p, got, oracle_encode(p, items, W))
    cu = got["cu_out"]
    for r in range(len(items)):
        alone = gpu_encode(p, [items[r]], W, enc=got["enc"], wdev=got["wdev"])
        np.testing.assert_array_equal(alone["out"], got["out"][cu[r]:cu[r + 1]])


def test_refused_calls_write_nothing_and_leave_the_handle_usable():
    import torch
    from paper_2609_31551_amd import eas
    p = C.with_layers(C.QWEN_IMAGE, 2)
    W = synth.make_weights(p, 0)
    items = [torch.from_numpy(a).cuda() for a in synth.make_items(p, 2, 0, shapes=[(2, 56, 56), (2, 84, 56)])]
    enc = eas.Encoder(p, max_tokens=1000, max_seqs=2)
    wdev = eas.upload_weights(enc.cfg, W)
    packed, cu, grid = enc.pack_microbatch(items)
    ref, ref_cu = enc.encode_microbatch(packed, cu, grid, wdev)
    torch.cuda.synchronize()
    ref = ref.cpu()

    out = torch.full(ref.shape, float("nan"), dtype=ref.dtype, device="cuda")
    refused = [
        ("empty micro-batch", [0], grid, eas.EAS_ERR_CAPACITY),
        ("more requests than max_seqs", [0, 16, 40, 56], [[1, 4, 4], [1, 6, 4], [1, 4, 4]], eas.EAS_ERR_CAPACITY),
        ("more tokens than max_tokens", [0, 1200], [[1, 30, 40]], eas.EAS_ERR_CAPACITY),
        ("grid does not match cu_seqlens", [0, 16, 40], [[1, 4, 4], [1, 4, 4]], eas.EAS_ERR_SHAPE),
    ]
    for what, bad_cu, bad_grid, status in refused:
        print("[edge] refused call: %s" % what, flush=True)
        with pytest.raises(eas.EasError) as ei:
            enc.encode_microbatch(packed, np.asarray(bad_cu, np.int32), np.asarray(bad_grid, np.int32), wdev, out=out)
        assert ei.value.status == status, (what, ei.value.status)
        torch.cuda.synchronize()
        assert torch.isnan(out).all().item(), what   # nothing was written
    again, again_cu = enc.encode_microbatch(packed, cu, grid, wdev, out=out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(again_cu, ref_cu)
    np.testing.assert_array_equal(again.cpu().numpy(), ref.numpy())


def test_mfma_rate_probe_reports_a_rate_within_the_clock_limit():
    """The measurement probe's flop count: 256 CUs x 4 SIMDs x one 32x32x16 MFMA
    (32768 flops) per 32 cycles at 2.4 GHz bound its rate from above; both
    operand kinds give a positive, finite rate below that bound."""
    import math
    from paper_2609_31551_amd import eas
    for zero in (False, True):
        print("[edge] mfma rate probe, zero operands=%s" % zero, flush=True)
        tf = eas.mfma_rate_probe(zero, iters=20000)
        assert math.isfinite(tf) and 50.0 < tf < 2.62e3, (zero, tf)

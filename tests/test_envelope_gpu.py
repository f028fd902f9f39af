"""Per-destination envelopes on the GPU (Section 3.3): the device gather is an
exact permutation of rows, and a micro-batch encoded in the planned order
already is the set of envelopes (bit-identical to gathering the
request-ordered output)."""
import numpy as np
import pytest

from _harness import gpu_encode
from paper_2609_31551_amd import configs as C
from paper_2609_31551_amd import router as R
from paper_2609_31551_amd import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dim,dtype", [(1024, "float32"), (3584, "bfloat16"), (4, "float32")])
def test_gather_is_an_exact_row_permutation(dim, dtype):
    import torch
    rng = np.random.default_rng(1)
    n, nd = 37, 3
    rows = rng.integers(0, 300, n)
    rows[5] = 0
    dest = rng.integers(0, nd, n)
    src_rows = np.concatenate([[0], np.cumsum(rows)])
    src = torch.randn(int(src_rows[-1]), dim, device="cuda").to(getattr(torch, dtype))
    order, dest_rows, req_rows = R.envelope_plan(dest, nd, rows)
    dst = torch.full_like(src, 7.0)
    print("[envelope] gather %d requests x %s %s" % (n, dim, dtype), flush=True)
    R.envelope_gather(src, src_rows, req_rows, dst)
    torch.cuda.synchronize()
    ref = torch.cat([src[src_rows[i]:src_rows[i + 1]] for i in order])
    assert torch.equal(dst, ref)


def test_planned_order_encodes_straight_into_envelopes():
    import torch
    p = C.with_layers(C.QWEN_IMAGE, 2)
    W = synth.make_weights(p, 0)
    items = synth.make_items(p, 5, 0, shapes=[(2, 224, 308), (2, 392, 224), (2, 280, 280), (2, 224, 224),
                                              (2, 336, 224)])
    dest = [1, 0, 1, 1, 0]
    batch = gpu_encode(p, items, W)
    cu = batch["cu_out"]
    rows = np.diff(cu)
    order, dest_rows, req_rows = R.envelope_plan(dest, 2, rows)
    src = torch.from_numpy(batch["out"]).cuda()
    dst = torch.empty_like(src)
    R.envelope_gather(src, cu, req_rows, dst)
    torch.cuda.synchronize()
    planned = gpu_encode(p, [items[i] for i in order], W, enc=batch["enc"], wdev=batch["wdev"])
    np.testing.assert_array_equal(planned["out"], dst.cpu().numpy())
    np.testing.assert_array_equal(planned["cu_out"], np.concatenate([[0], np.cumsum(rows[order])]))

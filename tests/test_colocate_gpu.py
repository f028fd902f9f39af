"""GPU checks of the compute-unit reservation behind the co-location profile
(include/eas_colocate.h, Section 3.4 dynamic SM partitioning): holding half of
the CUs slows a compute-bound encode (CLIP, 64 images) by roughly the lost
share and leaves its result bit-identical; a reservation ends when released
and, unreleased, at its time limit; out-of-range sizes are refused."""
import time

import pytest

pytestmark = pytest.mark.gpu


# Run in a fresh process with more hardware queues than streams: in the test
# process the many streams of earlier tests share HIP's default 4 queues, and a
# stream sharing the reservation's queue would wait for the reservation.
_HALF = """
import json
import torch
from paper_2609_31551_amd import colocate as K, configs as C, eas, synth
p = C.with_layers(C.CLIP_L336, 2)
n = 64
W = synth.make_weights(p, 0)
items = [torch.from_numpy(a).cuda() for a in synth.make_items(p, n, 0)]
enc = eas.Encoder(p, max_tokens=577 * n, max_seqs=n)
wdev = eas.upload_weights(enc.cfg, W)
out = torch.empty((577 * n, p["out_dim"]), dtype=torch.float32, device="cuda")
def run(stream):
    with torch.cuda.stream(stream):
        packed, cu, grid = enc.pack_microbatch(items, stream=stream)
        enc.encode_microbatch(packed, cu, grid, wdev, out=out, stream=stream)
t_full = K.encode_latency_ms(run, 1.0, reps=3)
ref = out.clone()
t_half = K.encode_latency_ms(run, 0.5, reps=3, max_s=5.0)
torch.cuda.synchronize()
print(json.dumps({"full": t_full, "half": t_half, "same": bool(torch.equal(out, ref))}))
"""


def test_holding_half_the_cus_slows_encode_and_keeps_its_result():
    import json
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ, GPU_MAX_HW_QUEUES="16", PYTHONPATH=root)
    r = subprocess.run([sys.executable, "-c", _HALF], env=env, cwd=root, capture_output=True, text=True, timeout=150)
    assert r.returncode == 0, r.stderr[-2000:]
    res = json.loads([l for l in r.stdout.splitlines() if l.startswith("{")][-1])
    print("[colocate] CLIP x64, 2 layers: %.3f ms whole device, %s ms on half" % (res["full"], res["half"]), flush=True)
    assert res["same"]
    assert res["half"] is not None, "encode stalled behind the reservation"
    assert 1.2 <= res["half"] / res["full"] <= 3.0, res


def test_reservation_ends_on_release_and_at_its_time_limit():
    import torch
    from paper_2609_31551_amd import colocate as K
    from paper_2609_31551_amd import eas
    t0 = time.time()
    with K.CuReservation(K.device_cus() // 2, max_s=10.0):
        pass
    assert time.time() - t0 < 2.0   # released on exit, long before its 10 s limit
    started = torch.zeros(16, dtype=torch.int32, pin_memory=True)
    release = torch.zeros(1, dtype=torch.int32, pin_memory=True)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    t0 = time.time()
    assert K.LIB.eas_cu_reserve(16, 0.3, started.data_ptr(), release.data_ptr(), s.cuda_stream) == eas.EAS_OK
    s.synchronize()
    elapsed = time.time() - t0
    print("[colocate] unreleased 0.3 s reservation ended after %.3f s" % elapsed, flush=True)
    assert int(started.sum()) == 16
    assert 0.25 <= elapsed <= 3.0, elapsed


def test_reservation_refuses_sizes_outside_the_device():
    import torch
    from paper_2609_31551_amd import colocate as K
    from paper_2609_31551_amd import eas
    started = torch.zeros(K.device_cus() + 1, dtype=torch.int32, pin_memory=True)
    release = torch.zeros(1, dtype=torch.int32, pin_memory=True)
    for n in (0, -1, K.reserve_max(K.device_cus()) + 1, K.device_cus() + 1):
        assert K.LIB.eas_cu_reserve(n, 1.0, started.data_ptr(), release.data_ptr(), None) == eas.EAS_ERR_INVALID_ARG
    assert int(started.sum()) == 0

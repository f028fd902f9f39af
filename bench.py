"""Encode-stage throughput on one MI355X.

A step is one pass of the whole Encode hot path over one micro-batch that is
already resident in HBM: pack the raw requests into a padding-free batch, then
run the encoder forward pass and connector (eas_pack_microbatch +
eas_encode_microbatch).  The headline workload is a micro-batch of 64 CLIP
ViT-L/14-336 images (577 tokens each, bf16 weights N(0, 0.02), pixels U[0,1),
seed 0), the image workload of the paper's Table 3.  Prints ONE JSON line.

Besides the headline, every workload of the evaluation (Section 4.1) is swept
over micro-batch sizes on a fixed pool of requests: a pass walks the whole
pool in consecutive micro-batches of size B, so every B encodes the same
requests (CLIP: 64 images; variable-resolution Qwen2-VL-style images: 64
images; video: 4 clips of 16 x 448 x 448; Whisper-style audio: 32 clips).

Roofline: during a second pass over the same steps every kernel launch is
bracketed by HIP events on the encoder's stream; the kernel with the largest
total time is the dominant kernel, and its algorithmic flops per launch over
its mean duration is compared with the bf16 dense MFMA peak.  The CPU
baseline times the fp64 reference on a bounded sample (whole images, full
depth) on the host cores, and on one request with one thread;
per-workload reference timings at micro-batch 1 run at reduced depth where
the full depth would exceed the time budget, and say so.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
METRIC = "encoded tokens/sec + images/sec vs micro-batch size; % bf16 MFMA peak (1 GPU)"
MFMA_KERNELS = ("gemm_", "attn_")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--preset", default="clip_vit_l14_336")
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--sweep", default="1,2,4,8,16,32,64", help="micro-batch sizes of the headline preset ('' to skip)")
    ap.add_argument("--workloads", default="qwen2vl_vit_image:64:1,2,4,8,16,32;qwen2vl_vit_video:4:1,2,4;"
                    "whisper_large_enc:32:1,2,4,8,16,32",
                    help="other workloads swept as preset:pool:sizes;... ('' to skip)")
    ap.add_argument("--cpu-configs-budget-s", type=float, default=8.0,
                    help="per-workload time budget of the micro-batch-1 reference timings (0 to skip)")
    ap.add_argument("--sweep-steps", type=int, default=5)
    ap.add_argument("--serving-s", type=float, default=3.0,
                    help="seconds of live Poisson arrivals replayed through the micro-batcher (0 to skip)")
    ap.add_argument("--serving-load", type=float, default=0.7,
                    help="offered load of the serving runs, as a fraction of the micro-batch-64 capacity")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the event-timed roofline pass")
    ap.add_argument("--colocation", default="",
                    help="micro-batch sizes of a co-location profile of the headline preset: encode latency "
                         "with 12.5/30/50/70/90%% of the CUs and the smallest-safe-share table ('' to skip)")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (HBM counter calibration)")
    return ap.parse_args()


def copy_calibration(mib):
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n * 4, "copy_calibration_bytes_written": n * 4}))


def mfma_power_probe(n=8192, reps=10):
    """The vendor library's bf16 matmul (torch.matmul -> hipBLASLt) at n^3 on
    normally distributed operands and on all-zero operands.  Same instructions,
    same memory traffic; only the operand bits differ, so the gap is what the
    board's power budget takes from MFMA throughput when the bits toggle.  Beside
    it, the library's register-only MFMA probe on random and zero operands."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(7)
    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16, generator=g)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16, generator=g)
    za, zb = torch.zeros_like(a), torch.zeros_like(b)
    out = {}
    for name, x, y in (("random", a, b), ("zero", za, zb)):
        for _ in range(3):
            torch.matmul(x, y)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            torch.matmul(x, y)
        e1.record()
        torch.cuda.synchronize()
        out[name + "_tflops"] = 2.0 * n ** 3 * reps / (e0.elapsed_time(e1) * 1e-3) / 1e12
    out["op"] = "torch.matmul bf16 %d x %d x %d, %d launches back to back" % (n, n, n, reps)
    out["zero_over_random"] = out["zero_tflops"] / out["random_tflops"]
    # the MFMA issue rate alone: operands in registers, no memory traffic
    from paper_2609_31551_amd import eas
    out["register_only_random_tflops"] = eas.mfma_rate_probe(False)
    out["register_only_zero_tflops"] = eas.mfma_rate_probe(True)
    del a, b, za, zb
    torch.cuda.empty_cache()
    return out


# kernel name -> the sources that decide what it reads and writes per launch
TRAFFIC_SOURCES = {
    "gemm_bf16_256x256": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_128x128": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_async_256x256": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_async_res_256x256": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_async_res_256x128": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_async_res_128x128": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_async_256x128": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_async_128x128": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_64x64": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "gemm_bf16_64x128": ("gemm_bf16.hip", "common.h", "eas_api.cpp"),
    "attn_bf16_hd64": ("attention_dma.hip", "common.h", "eas_api.cpp"),
    "attn_bf16_hd80": ("attention_dma.hip", "common.h", "eas_api.cpp"),
    "attn_bf16_hd80_q256": ("attention_dma.hip", "common.h", "eas_api.cpp"),
    "ln_apply_bf16": ("elementwise.hip", "common.h", "eas_api.cpp"),
    "rope": ("elementwise.hip", "common.h", "eas_api.cpp"),
}


def traffic_record(workload, kernel):
    """HBM bytes per launch of `kernel` on `workload` (a preset name and
    micro-batch size, "clip_vit_l14_336/64") from the committed counter
    summary, if it was taken on the current sources of that kernel."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path) or kernel not in TRAFFIC_SOURCES:
        return None
    rec = json.load(open(path)).get(workload, {}).get(kernel)
    if not rec:
        return None
    if rec.get("source_sha") != source_sha(TRAFFIC_SOURCES[kernel]):
        return None
    return rec.get("bytes_per_launch")


def source_sha(files):
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_31551_amd", "csrc")
    for f in files:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


class Workload:
    """A pool of synthetic requests resident in HBM, walked in micro-batches."""

    def __init__(self, preset, pool, max_batch, seed=0):
        import torch
        from paper_2609_31551_amd import eas, synth
        self.preset, self.pool = preset, pool
        t0 = time.time()
        self.weights_host = synth.make_weights(preset, seed)
        self.items_host = synth.make_items(preset, pool, seed)
        self.gen_s = time.time() - t0
        cfg = eas.make_config(preset, 1 << 18, 1)   # shape queries only
        tchw = [list(a.shape) if a.ndim == 4 else [1, 1] + list(a.shape) for a in self.items_host]
        self.item_tokens = [int(eas.microbatch_shape(cfg, [t])[0][-1]) for t in tchw]
        max_tokens = sum(sorted(self.item_tokens)[-max_batch:])
        self.stream = torch.cuda.Stream()
        self.enc = eas.Encoder(preset, max_tokens=max_tokens, max_seqs=max_batch)
        self.wdev = eas.upload_weights(self.enc.cfg, self.weights_host)
        self.items = [torch.from_numpy(a).cuda() for a in self.items_host]
        self.whisper = preset["kind"] == "whisper"
        item_rows = [self.enc.out_rows([0, t]) for t in self.item_tokens]
        rows = sum(sorted(item_rows)[-max_batch:])
        self.out = torch.empty((rows, preset["out_dim"]), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()

    def step(self, start, n):
        """Pack + encode requests [start, start + n)."""
        import torch
        with torch.cuda.stream(self.stream):
            packed, cu, grid = self.enc.pack_microbatch(self.items[start:start + n], stream=self.stream)
            self.enc.encode_microbatch(packed, cu, None if self.whisper else grid, self.wdev,
                                       out=self.out[:self.enc.out_rows(cu)], stream=self.stream)
        return int(cu[-1])

    def run_pass(self, b, first=None):
        """Consecutive micro-batches of b over the first `first` requests (default: the pool)."""
        end = self.pool if first is None else first
        tok = 0
        for i in range(0, end, b):
            tok += self.step(i, min(b, end - i))
        return tok

    def time_passes(self, b, reps, warmup, first=None):
        import torch
        for _ in range(warmup):
            self.run_pass(b, first)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(self.stream)
        tok = 0
        for _ in range(reps):
            tok += self.run_pass(b, first)
        t1.record(self.stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / reps, tok / reps

    def profile_passes(self, b, reps, first=None):
        import torch
        self.enc.profile_read()
        self.enc.profile_enable(True)
        for _ in range(reps):
            self.run_pass(b, first)
        torch.cuda.synchronize()
        self.enc.profile_enable(False)
        return self.enc.profile_read()

    def close(self):
        import torch
        torch.cuda.synchronize()
        self.enc.close()
        del self.items, self.wdev, self.out
        torch.cuda.empty_cache()


def mfma_fraction(prof):
    fl = sum(v["flops"] for k, v in prof.items() if k.startswith(MFMA_KERNELS))
    ms = sum(v["ms"] for k, v in prof.items() if k.startswith(MFMA_KERNELS))
    return (fl / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS) if ms > 0 else None


def sweep_rows(wl, sizes, reps, profile):
    """Throughput of one pass over the pool at each micro-batch size."""
    rows = []
    for b in sizes:
        ms, tok = wl.time_passes(b, reps, 1)
        row = {"micro_batch": b, "tokens_per_s": tok / (ms * 1e-3), "items_per_s": wl.pool / (ms * 1e-3),
               "ms_per_pass": ms, "micro_batches_per_pass": -(-wl.pool // b)}
        if profile:
            prof = wl.profile_passes(b, 1)
            fl = sum(v["flops"] for v in prof.values())
            row["gemm_attn_mfma_frac"] = mfma_fraction(prof)
            row["whole_call_mfma_frac"] = fl / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS
            if b == max(sizes):
                row["kernels"] = kernel_table(prof, 1)
        rows.append(row)
    return rows


def kernel_table(prof, passes):
    """Per-kernel time per pass, share, algorithmic bytes and flops per launch,
    and TFLOP/s (MFMA kernels) or GB/s."""
    total_ms = sum(v["ms"] for v in prof.values())
    return {k: {"ms_per_step": v["ms"] / passes, "share": v["ms"] / total_ms,
                "launches_per_step": v["launches"] / passes,
                "alg_bytes_per_launch": v["bytes"] / v["launches"],
                "alg_flops_per_launch": v["flops"] / v["launches"],
                "tflops" if k.startswith(MFMA_KERNELS) else "gbs":
                    (v["flops"] / (v["ms"] * 1e-3) / 1e12) if k.startswith(MFMA_KERNELS)
                    else (v["bytes"] / (v["ms"] * 1e-3) / 1e9)}
            for k, v in sorted(prof.items(), key=lambda kv: -kv[1]["ms"])}


def oracle_threads():
    from threadpoolctl import threadpool_info
    return max([p.get("num_threads", 1) for p in threadpool_info()] + [1])


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(preset, wl, batch, budget_s):
    from oracle import encoder as O
    t0 = time.time()
    n_items, tokens = 0, 0
    while n_items < batch:
        item = wl.items_host[n_items]
        packed, cu, grid = O.pack(preset, [item])
        O.encode(preset, wl.weights_host, packed, cu, grid)
        n_items += 1
        tokens += int(cu[-1])
        if time.time() - t0 >= budget_s:
            break
    dt = time.time() - t0
    return {"value": tokens / dt, "unit": "tokens/s", "cores": oracle_threads(), "kind": "oracle",
            "sample": "%d of the %d requests, full %d-layer depth, float64, one request per call "
                      "(%.1f s)" % (n_items, batch, preset["layers"], dt),
            "items_per_s": n_items / dt, "cpu_model": cpu_model()}


def cpu_config_timing(preset, wl, budget_s):
    """The reference on the pool's first request (micro-batch 1).  Full depth
    when a one-layer run says it fits the budget; otherwise one- and two-layer
    runs, whose difference gives the per-layer time, and a full-depth
    estimate from them."""
    from paper_2609_31551_amd import configs as C
    from oracle import encoder as O
    packed, cu, grid = O.pack(preset, [wl.items_host[0]])
    tokens = int(cu[-1])

    def run(layers):
        t0 = time.time()
        O.encode(C.with_layers(preset, layers), wl.weights_host, packed, cu, grid)
        return time.time() - t0

    t1 = run(1)
    rec = {"micro_batch": 1, "tokens": tokens, "cores": oracle_threads()}
    if t1 * preset["layers"] <= budget_s:
        tf = run(preset["layers"]) if preset["layers"] > 1 else t1
        rec.update(depth=preset["layers"], seconds=tf, tokens_per_s=tokens / tf, measured_full_depth=True)
        return rec
    t2 = run(2)
    per_layer = max(t2 - t1, 1e-9)
    est = (t1 - per_layer) + preset["layers"] * per_layer
    rec.update(depth=2, seconds=t2, tokens_per_s_at_depth=tokens / t2, per_layer_s=per_layer,
               full_depth_estimate_s=est, tokens_per_s=tokens / est, measured_full_depth=False)
    return rec


def cpu_one_thread(preset, wl):
    """The reference on the pool's first request, full depth, with its BLAS
    held to one thread (timed directly: each call converts every layer's
    weights to float64, a fixed cost that drowns depth differences)."""
    from threadpoolctl import threadpool_limits
    from oracle import encoder as O
    packed, cu, grid = O.pack(preset, [wl.items_host[0]])
    tokens = int(cu[-1])
    with threadpool_limits(limits=1):
        t0 = time.time()
        O.encode(preset, wl.weights_host, packed, cu, grid)
        dt = time.time() - t0
    return {"micro_batch": 1, "tokens": tokens, "cores": 1, "depth": preset["layers"], "seconds": dt,
            "tokens_per_s": tokens / dt, "measured_full_depth": True}


def service_times(rows, pool, bound):
    """Seconds per micro-batch of b requests, b = 1 .. bound, from the swept
    pass times (linear between measured sizes)."""
    bs = [r["micro_batch"] for r in rows]
    per = [r["ms_per_pass"] * 1e-3 / r["micro_batches_per_pass"] for r in rows]
    return [0.0] + [float(v) for v in __import__("numpy").interp(range(1, bound + 1), bs, per)]


def colocation(wl, sizes, reps=3):
    """Encode latency of one pack + encode micro-batch against the share of the
    CUs left to it (Section 3.4, dynamic SM partitioning), and the table of the
    largest batch size each share sustains within 20% of exclusive access."""
    from paper_2609_31551_amd import colocate as K

    def run_for(b):
        def run(stream):
            wl.stream = stream
            wl.step(0, b)
        return run
    keep = wl.stream
    log = lambda m: print("[colocation] " + m, file=sys.stderr, flush=True)
    exclusive, latency = K.profile(run_for, sizes, K.LEVELS, reps, max_s=3.0, log=log)
    wl.stream = keep
    table = K.safe_share_table(latency, exclusive)
    return {"levels": list(K.LEVELS), "micro_batches": list(sizes), "threshold": K.THRESHOLD,
            "reps": reps, "cus": K.device_cus(),
            "exclusive_ms": {str(b): exclusive[b] for b in sizes},
            "latency_ms": {str(lv): {str(b): latency[lv][b] for b in sizes} for lv in K.LEVELS},
            "largest_safe_batch": {str(lv): table[lv] for lv in K.LEVELS},
            "share_for_batch": {str(b): K.select_share(table, b) for b in sizes},
            "mechanism": "CUs held by a reservation kernel (one workgroup per CU) while encode runs on the rest"}


def serving(wl, rows, load, live_s, B=64, p=0.6, max_age=1.0):
    """The Poisson-gap micro-batcher (Section 3.2) in front of this encoder.

    * replay cost of the library's batcher per arrival (C++);
    * four dispatch policies on one Poisson trace (the comparison of the
      paper's Figure 5), and the Poisson-gap rule under Gamma arrivals of CV
      0.5, 1, 2 (Section 4.5's sensitivity study), through a single encode
      server that takes the measured micro-batch times;
    * a live replay: Poisson arrivals at the same load drive the GPU encoder
      in real time; latency = batch completion (HIP event) - arrival."""
    import numpy as np
    import torch
    from paper_2609_31551_amd import batcher as L, synth
    svc = service_times(rows, wl.pool, B)
    capacity = B / svc[B]
    lam = load * capacity
    out = {"batch_bound": B, "fill_prob": p, "max_age_s": max_age, "capacity_items_per_s": capacity,
           "offered_items_per_s": lam, "gap_s": L.poisson_gap_threshold(B, p, lam)}

    arr = synth.arrival_trace(1000000, lam, 1.0, seed=0)
    t0 = time.perf_counter()
    L.batcher_simulate(arr, B, p, lam, max_age, svc)
    out["replay_ns_per_arrival"] = (time.perf_counter() - t0) / arr.shape[0] * 1e9

    def summarize(arr, r):
        lat = r["done_t"] - arr
        span = r["done_t"].max() - arr[0]
        return {"items_per_s": arr.shape[0] / span, "latency_mean_ms": float(lat.mean() * 1e3),
                "latency_p99_ms": float(np.percentile(lat, 99) * 1e3),
                "mean_batch": float(arr.shape[0] / r["n_batches"]), "batches": int(r["n_batches"])}

    arr = synth.arrival_trace(20000, lam, 1.0, seed=1)
    never = 1.0 - 1e-12       # p -> 1: the idle-gap condition never fires
    policies = {"fixed_bound_no_timeout": (never, 1e9), "timeout_2ms": (never, 0.002),
                "timeout_50ms": (never, 0.05), "poisson_gap": (p, max_age)}
    out["policies_cv1"] = {k: summarize(arr, L.batcher_simulate(arr, B, pp, lam, a, svc))
                           for k, (pp, a) in policies.items()}
    out["poisson_gap_vs_cv"] = {}
    for cv in (0.5, 1.0, 2.0):
        arr = synth.arrival_trace(20000, lam, cv, seed=2)
        out["poisson_gap_vs_cv"]["cv%.1f" % cv] = summarize(arr, L.batcher_simulate(arr, B, p, lam, max_age, svc))

    # deficit-counter router (Section 3.3): cost per decision, and the device
    # gather of the micro-batch's output into per-destination envelopes
    from paper_2609_31551_amd import router as R
    rt = R.Router(0.7)
    t0 = time.perf_counter()
    rt.route(1000000)
    out["router_ns_per_decision"] = (time.perf_counter() - t0) / 1e6 * 1e9
    n_req = wl.pool
    rows = np.array([wl.enc.out_rows([0, t]) for t in wl.item_tokens[:n_req]], np.int64)
    src_rows = np.concatenate([[0], np.cumsum(rows)])
    dest = rt.route(n_req).astype(np.int32)
    _, _, req_rows = R.envelope_plan(dest, 2, rows)
    src = wl.out[:int(src_rows[-1])]
    dst = torch.empty_like(src)
    with torch.cuda.stream(wl.stream):
        for _ in range(3):
            R.envelope_gather(src, src_rows, req_rows, dst, stream=wl.stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(wl.stream)
        for _ in range(20):
            R.envelope_gather(src, src_rows, req_rows, dst, stream=wl.stream)
        e1.record(wl.stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 20
    nbytes = 2 * src.numel() * src.element_size()
    out["envelope_gather"] = {"requests": n_req, "bytes_moved": nbytes, "ms": ms, "gbs": nbytes / (ms * 1e-3) / 1e9,
                              "roofline_frac": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
                              "note": "encoding in the planned order produces the envelopes with no copy"}

    if live_s > 0:
        arr = synth.arrival_trace(max(1, int(lam * live_s)), lam, 1.0, seed=3)
        bt = L.Batcher(B, p, lam, max_age)
        recs = []

        def dispatch():
            ids, _ = bt.take()
            items = [wl.items[j % wl.pool] for j in ids]
            with torch.cuda.stream(wl.stream):
                packed, cu, grid = wl.enc.pack_microbatch(items, stream=wl.stream)
                wl.enc.encode_microbatch(packed, cu, None if wl.whisper else grid, wl.wdev,
                                         out=wl.out[:wl.enc.out_rows(cu)], stream=wl.stream)
                ev = torch.cuda.Event(enable_timing=True)
                ev.record(wl.stream)
            recs.append((ids, ev))

        torch.cuda.synchronize()
        ev0 = torch.cuda.Event(enable_timing=True)
        ev0.record(wl.stream)
        start = time.perf_counter()
        i, n = 0, arr.shape[0]
        while i < n or bt.size():
            now = time.perf_counter() - start
            while i < n and arr[i] <= now:
                if bt.size() and bt.deadline() < arr[i]:
                    dispatch()
                if bt.arrive(arr[i], i):
                    dispatch()
                i += 1
            if bt.size() and bt.poll(now):
                dispatch()
        torch.cuda.synchronize()
        done = np.empty(n)
        for ids, ev in recs:
            done[ids] = ev0.elapsed_time(ev) * 1e-3
        r = {"done_t": done, "n_batches": len(recs)}
        out["live_poisson"] = dict(summarize(arr, r), seconds=float(arr[-1]), requests=int(n))
    return out


def parse_workloads(spec):
    out = []
    for part in spec.split(";"):
        part = part.strip()
        if not part:
            continue
        name, pool, sizes = part.split(":")
        out.append((name, int(pool), [int(b) for b in sizes.split(",") if b.strip()]))
    return out


def main():
    args = parse()
    if args.colocation:
        # the co-location profile runs a reservation beside the encoder's two streams: with
        # HIP's default of 4 hardware queues per process, streams share queues and run in
        # order, so encode work could sit behind the reservation (set before HIP starts)
        os.environ["GPU_MAX_HW_QUEUES"] = "16"
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (requests shard by "
              "micro-batch across independent encoders); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.copy_calib_mib:
        copy_calibration(args.copy_calib_mib)
        return
    import torch
    from paper_2609_31551_amd import configs as C
    preset = C.PRESETS[args.preset]
    torch.cuda.set_device(0)
    sweep = [int(b) for b in args.sweep.split(",") if b.strip()]
    pool = max([args.batch] + sweep)
    wl = Workload(preset, pool, pool)

    ms, tok = wl.time_passes(args.batch, args.steps, args.warmup, first=args.batch)
    result = {
        "metric": METRIC, "value": tok / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": preset["dtype"], "data": "synthetic",
        "config": {"workload": "%s encoder, micro-batch of %d requests (%d tokens), pack + encode"
                               % (preset["name"], args.batch, tok),
                   "micro_batch": args.batch, "tokens_per_step": tok, "layers": preset["layers"],
                   "hidden": preset["hidden"], "parallelism": "single GPU"},
        "images_per_s": args.batch / (ms * 1e-3),
    }
    if not args.no_profile:
        prof = wl.profile_passes(args.batch, args.steps, first=args.batch)
        dom = max(prof, key=lambda k: prof[k]["ms"])
        p = prof[dom]
        is_mfma = dom.startswith(MFMA_KERNELS)
        per_launch_ms = p["ms"] / p["launches"]
        if is_mfma:
            achieved = p["flops"] / p["launches"] / (per_launch_ms * 1e-3) / 1e12
            peak, unit = PEAK_BF16_TFLOPS, "TFLOP/s"
        else:
            achieved = p["bytes"] / p["launches"] / (per_launch_ms * 1e-3) / 1e9
            peak, unit = PEAK_HBM_GBS, "GB/s"
        result["roofline"] = {"bound": "mfma" if is_mfma else "hbm", "kernel": dom, "achieved": achieved,
                              "peak": peak, "unit": unit, "frac": achieved / peak,
                              "traffic": traffic_record("%s/%d" % (args.preset, args.batch), dom),
                              "traffic_unit": "HBM bytes per launch",
                              "mean_launch_ms": per_launch_ms,
                              "launches_per_step": p["launches"] / args.steps}
        result["kernels"] = kernel_table(prof, args.steps)
        result["gemm_attn_mfma_frac"] = mfma_fraction(prof)
        result["mfma_power_probe"] = mfma_power_probe()
    workloads = {}
    if sweep:
        workloads[preset["name"]] = {"pool": pool, "sweep": sweep_rows(wl, sweep, args.sweep_steps,
                                                                       not args.no_profile)}
    doubling = [1 << i for i in range(max(sweep).bit_length())] if sweep else []
    if len(doubling) > 1 and set(doubling) <= set(sweep):
        from paper_2609_31551_amd import capacity as K
        rows = {r["micro_batch"]: r["items_per_s"] for r in workloads[preset["name"]]["sweep"]}
        c_e, b_sat, curve = K.saturation_capacity(lambda b: rows[b], doubling[-1])
        lam = args.serving_load * c_e
        result["capacity"] = {"c_e_items_per_s": c_e, "b_sat": b_sat, "curve": curve,
                              "rule": "double B until a doubling gains < 5% (Section 3.1)",
                              "example_load_items_per_s": lam, "rho_e": K.utilization(lam, 1, c_e),
                              "b_max": K.batch_cap(lam, 1)}
    if sweep and args.serving_s >= 0 and max(sweep) == pool and len(sweep) > 1:
        result["serving"] = serving(wl, workloads[preset["name"]]["sweep"], args.serving_load, args.serving_s,
                                    B=pool)
    if args.colocation:
        sizes = [int(b) for b in args.colocation.split(",") if b.strip()]
        if max(sizes) > pool:
            raise SystemExit("--colocation sizes must not exceed the pool (%d)" % pool)
        result["colocation"] = colocation(wl, sizes)
    cpu_configs = {}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(preset, wl, args.batch, args.cpu_budget_s)
        result["cpu_baseline"]["one_thread"] = cpu_one_thread(preset, wl)
        if args.cpu_configs_budget_s > 0:
            cpu_configs[preset["name"]] = cpu_config_timing(preset, wl, args.cpu_configs_budget_s)
    wl.close()
    for name, wpool, sizes in parse_workloads(args.workloads):
        other = Workload(C.PRESETS[name], wpool, max(sizes))
        workloads[name] = {"pool": wpool, "pool_tokens": sum(other.item_tokens),
                           "sweep": sweep_rows(other, sizes, args.sweep_steps, not args.no_profile)}
        if not args.no_cpu_baseline and args.cpu_configs_budget_s > 0:
            cpu_configs[name] = cpu_config_timing(C.PRESETS[name], other, args.cpu_configs_budget_s)
        other.close()
        print("[bench] %s swept" % name, file=sys.stderr, flush=True)
    if workloads:
        result["workloads"] = workloads
    if cpu_configs:
        result["cpu_configs"] = cpu_configs
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()

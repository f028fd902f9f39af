"""Encode-stage throughput on one MI355X.

A step is one pass of the whole Encode hot path over one micro-batch that is
already resident in HBM: pack the raw requests into a padding-free batch, then
run the encoder forward pass and connector (eas_pack_microbatch +
eas_encode_microbatch).  The default workload is a micro-batch of 64 CLIP
ViT-L/14-336 images (577 tokens each, bf16 weights N(0, 0.02), pixels U[0,1),
seed 0), the image workload of the paper's Table 3; a sweep over micro-batch
sizes 1, 8, 32 and 64 follows.  Prints ONE JSON line.

Roofline: during a second pass over the same steps every kernel launch is
bracketed by HIP events on the encoder's stream; the kernel with the largest
total time is the dominant kernel, and its algorithmic flops per launch over
its mean duration is compared with the bf16 dense MFMA peak.  The CPU
baseline times the fp64 reference on a bounded sample (whole images, full
depth) on the host cores.
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
    ap.add_argument("--sweep", default="1,8,32,64", help="micro-batch sizes ('' to skip)")
    ap.add_argument("--sweep-steps", type=int, default=5)
    ap.add_argument("--cpu-budget-s", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip the event-timed roofline pass")
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


def traffic_record(kernel):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(kernel)
    if not rec:
        return None
    if rec.get("source_sha") != source_sha():
        return None
    return rec.get("bytes_per_launch")


def source_sha():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_31551_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


class Workload:
    def __init__(self, preset, batch, seed=0):
        import torch
        from paper_2609_31551_amd import eas, synth
        self.preset, self.batch = preset, batch
        t0 = time.time()
        self.weights_host = synth.make_weights(preset, seed)
        self.items_host = synth.make_items(preset, batch, seed)
        self.gen_s = time.time() - t0
        tchw = [list(a.shape) if a.ndim == 4 else [1, 1] + list(a.shape) for a in self.items_host]
        cu, _, _, _ = eas.microbatch_shape(eas.make_config(preset, 1 << 30, batch), tchw)
        self.tokens = int(cu[-1])
        self.stream = torch.cuda.Stream()
        self.enc = eas.Encoder(preset, max_tokens=self.tokens, max_seqs=batch)
        self.wdev = eas.upload_weights(self.enc.cfg, self.weights_host)
        self.items = [torch.from_numpy(a).cuda() for a in self.items_host]
        self.packed, self.cu, self.grid = self.enc.pack_microbatch(self.items, stream=self.stream)
        self.grid_arg = None if preset["kind"] == "whisper" else self.grid
        self.out = torch.empty((self.enc.out_rows(self.cu), preset["out_dim"]), dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()

    def step(self, n):
        """One pass over the first n requests: pack + encode."""
        import torch
        with torch.cuda.stream(self.stream):
            packed, cu, grid = self.enc.pack_microbatch(self.items[:n], stream=self.stream)
            self.enc.encode_microbatch(packed, cu, grid if self.grid_arg is not None else None, self.wdev,
                                       out=self.out[:self.enc.out_rows(cu)], stream=self.stream)
        return int(cu[-1])

    def time_steps(self, n, steps, warmup):
        import torch
        for _ in range(warmup):
            self.step(n)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(self.stream)
        tok = 0
        for _ in range(steps):
            tok += self.step(n)
        t1.record(self.stream)
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1)
        return ms / steps, tok / steps

    def profile_steps(self, n, steps):
        import torch
        self.enc.profile_read()
        self.enc.profile_enable(True)
        for _ in range(steps):
            self.step(n)
        torch.cuda.synchronize()
        self.enc.profile_enable(False)
        return self.enc.profile_read()


def mfma_fraction(prof):
    fl = sum(v["flops"] for k, v in prof.items() if k.startswith(MFMA_KERNELS))
    ms = sum(v["ms"] for k, v in prof.items() if k.startswith(MFMA_KERNELS))
    return (fl / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS) if ms > 0 else None


def cpu_baseline(preset, wl, budget_s):
    import numpy as np
    from threadpoolctl import threadpool_info
    from oracle import encoder as O
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    t0 = time.time()
    n_items, tokens = 0, 0
    while n_items < wl.batch:
        item = wl.items_host[n_items]
        packed, cu, grid = O.pack(preset, [item])
        O.encode(preset, wl.weights_host, packed, cu, grid)
        n_items += 1
        tokens += int(cu[-1])
        if time.time() - t0 >= budget_s:
            break
    dt = time.time() - t0
    return {"value": tokens / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": "%d of the %d requests, full %d-layer depth, float64, one request per call "
                      "(%.1f s)" % (n_items, wl.batch, preset["layers"], dt),
            "items_per_s": n_items / dt}


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (requests shard by "
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
    wl = Workload(preset, max([args.batch] + sweep))

    ms, tok = wl.time_steps(args.batch, args.steps, args.warmup)
    items_per_s = args.batch / (ms * 1e-3)
    result = {
        "metric": METRIC, "value": tok / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": preset["dtype"], "data": "synthetic",
        "config": {"workload": "%s encoder, micro-batch of %d requests (%d tokens), pack + encode"
                               % (preset["name"], args.batch, tok),
                   "micro_batch": args.batch, "tokens_per_step": tok, "layers": preset["layers"],
                   "hidden": preset["hidden"], "parallelism": "single GPU"},
        "images_per_s": items_per_s,
    }
    if not args.no_profile:
        prof = wl.profile_steps(args.batch, args.steps)
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
                              "traffic": traffic_record(dom), "mean_launch_ms": per_launch_ms,
                              "launches_per_step": p["launches"] / args.steps}
        total_ms = sum(v["ms"] for v in prof.values())
        result["kernels"] = {k: {"ms_per_step": v["ms"] / args.steps, "share": v["ms"] / total_ms,
                                 "tflops" if k.startswith(MFMA_KERNELS) else "gbs":
                                     (v["flops"] / (v["ms"] * 1e-3) / 1e12) if k.startswith(MFMA_KERNELS)
                                     else (v["bytes"] / (v["ms"] * 1e-3) / 1e9)}
                             for k, v in sorted(prof.items(), key=lambda kv: -kv[1]["ms"])}
        result["gemm_attn_mfma_frac"] = mfma_fraction(prof)
    if sweep:
        rows = []
        for b in sweep:
            ms_b, tok_b = wl.time_steps(b, args.sweep_steps, 2)
            row = {"micro_batch": b, "tokens_per_s": tok_b / (ms_b * 1e-3), "items_per_s": b / (ms_b * 1e-3),
                   "ms_per_step": ms_b}
            if not args.no_profile:
                row["gemm_attn_mfma_frac"] = mfma_fraction(wl.profile_steps(b, args.sweep_steps))
            rows.append(row)
        result["sweep"] = rows
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(preset, wl, args.cpu_budget_s)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()

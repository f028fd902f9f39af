"""Seeded synthetic weights and inputs (numpy only; no encoder arithmetic).

This module is the one place that both the fp64 reference and the HIP path
take their inputs from.  It draws numbers and rounds them to the storage
precision of a preset; it computes nothing the encoder computes.

Weights: tensor i of ``weight_specs(cfg)`` is drawn by PCG64 from the i-th
child of ``SeedSequence(seed)``; linear weights, biases, CLS and position
tables are N(0, 0.02), LayerNorm gains are 1 and offsets 0.  Values are then
rounded to bfloat16 (round-to-nearest-even) for bf16 presets and kept as
float32 arrays holding bf16-representable values, so that both sides consume
exactly the same numbers.

Inputs: a second generator, PCG64(seed + 1), draws image sizes first (for the
variable-resolution preset) and then the pixels of each item in order:
U[0, 1) pixels for images and clips, N(0, 1) log-mel features for audio.
"""
import numpy as np

from . import configs as C


def round_to_bf16(a):
    """Round float32 values to the nearest bfloat16 (ties to even); finite inputs."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    u = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return u.view(np.float32).reshape(a.shape)


def to_bf16_bits(a):
    """float32 array of bf16-representable values -> uint16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    return (a.view(np.uint32) >> 16).astype(np.uint16)


def bf16_bits_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def weight_specs(cfg):
    """Canonical tensor list: (name, shape, init) in draw order.

    Linear weights are [out, in] row-major.  ``init`` is "normal", "ones" or
    "zeros".
    """
    d, f, L = cfg["hidden"], cfg["mlp"], cfg["layers"]
    kind = cfg["kind"]
    specs = []
    if kind == C.KIND_WHISPER:
        nm = cfg["n_mels"]
        specs += [("conv1.w", (d, nm * 3), "normal"), ("conv1.b", (d,), "normal"),
                  ("conv2.w", (d, d * 3), "normal"), ("conv2.b", (d,), "normal")]
    else:
        specs += [("patch.w", (d, C.k_patch(cfg)), "normal"), ("patch.b", (d,), "normal")]
    gh, gw = cfg["pos_grid"]
    if kind == C.KIND_VIT_CLS_ABS:
        specs += [("cls", (d,), "normal"), ("pos", (1 + gh * gw, d), "normal"),
                  ("ln_pre.g", (d,), "ones"), ("ln_pre.b", (d,), "zeros")]
    elif kind == C.KIND_VIT_ABS:
        specs += [("pos", (gh * gw, d), "normal")]
    for i in range(L):
        p = "layers.%d." % i
        specs += [(p + "ln1.g", (d,), "ones"), (p + "ln1.b", (d,), "zeros"),
                  (p + "qkv.w", (3 * d, d), "normal"), (p + "qkv.b", (3 * d,), "normal"),
                  (p + "o.w", (d, d), "normal"), (p + "o.b", (d,), "normal"),
                  (p + "ln2.g", (d,), "ones"), (p + "ln2.b", (d,), "zeros"),
                  (p + "fc1.w", (f, d), "normal"), (p + "fc1.b", (f,), "normal"),
                  (p + "fc2.w", (d, f), "normal"), (p + "fc2.b", (d,), "normal")]
    if cfg["merge"] == 2:
        m, o = 4 * d, cfg["out_dim"]
        specs += [("ln_q.g", (d,), "ones"), ("ln_q.b", (d,), "zeros"),
                  ("m1.w", (m, m), "normal"), ("m1.b", (m,), "normal"),
                  ("m2.w", (o, m), "normal"), ("m2.b", (o,), "normal")]
    if kind == C.KIND_WHISPER:
        specs += [("ln_post.g", (d,), "ones"), ("ln_post.b", (d,), "zeros")]
    return specs


def _draw_tensor(seed_seq, shape, init, std, bf16):
    if init == "normal":
        rng = np.random.Generator(np.random.PCG64(seed_seq))
        a = rng.standard_normal(int(np.prod(shape)), dtype=np.float32) * np.float32(std)
        a = a.reshape(shape)
    elif init == "ones":
        a = np.ones(shape, np.float32)
    else:
        a = np.zeros(shape, np.float32)
    return round_to_bf16(a) if bf16 else a


def make_weights(cfg, seed=0, std=0.02, threads=8):
    """Dict name -> float32 array.

    Tensor i of ``weight_specs`` is drawn from its own PCG64 stream, the i-th
    child of ``SeedSequence(seed)``, so tensors can be drawn in parallel and
    every tensor's values are fixed by (seed, i) alone.
    """
    from concurrent.futures import ThreadPoolExecutor
    specs = weight_specs(cfg)
    kids = np.random.SeedSequence(seed).spawn(len(specs))
    bf16 = cfg["dtype"] == "bf16"
    with ThreadPoolExecutor(max_workers=threads) as ex:
        arrays = list(ex.map(lambda i: _draw_tensor(kids[i], specs[i][1], specs[i][2], std, bf16),
                             range(len(specs))))
    return {spec[0]: a for spec, a in zip(specs, arrays)}


QWEN_SIDES = tuple(range(224, 1344 + 1, 28))   # the 41 multiples of 28 in [224, 1344]


def qwen_image_sizes(rng, n):
    """Draw (H, W): each side uniform over QWEN_SIDES, keep only 0.5 <= W/H <= 2."""
    sizes = []
    while len(sizes) < n:
        h = QWEN_SIDES[int(rng.integers(0, len(QWEN_SIDES)))]
        w = QWEN_SIDES[int(rng.integers(0, len(QWEN_SIDES)))]
        if 0.5 <= w / h <= 2.0:
            sizes.append((h, w))
    return sizes


def default_item_shape(cfg):
    """(frames, H, W) of one item of the preset's workload (vision presets)."""
    name = cfg["name"].split("_L")[0]
    if cfg["kind"] == C.KIND_VIT_ABS:
        return (1, 56, 56)
    if cfg["kind"] == C.KIND_VIT_CLS_ABS:
        return (1, 336, 336)
    if name.startswith("qwen2vl_vit_video"):
        return (16, 448, 448)
    return None   # variable-resolution images: drawn per item


def make_items(cfg, n, seed=0, shapes=None):
    """n raw inputs of the preset's workload.

    Vision: float32 arrays [frames, C, H, W] with U[0,1) pixels; the
    variable-resolution preset duplicates each image into 2 identical frames.
    Audio: float32 arrays [n_mels, n_frames] with N(0,1) values.
    ``shapes`` (list of (frames, H, W)) overrides the preset's item shapes.
    """
    rng = np.random.Generator(np.random.PCG64(seed + 1))
    items = []
    if cfg["kind"] == C.KIND_WHISPER:
        for _ in range(n):
            items.append(rng.standard_normal((cfg["n_mels"], cfg["n_frames"]), dtype=np.float32))
    else:
        if shapes is None:
            fixed = default_item_shape(cfg)
            if fixed is None:
                shapes = [(cfg["temporal_patch"], h, w) for h, w in qwen_image_sizes(rng, n)]
            else:
                shapes = [fixed] * n
        dup = cfg["kind"] == C.KIND_VIT_ROPE and cfg["rope_sections"][0] == 0
        for (t, h, w) in shapes:
            if dup:
                one = rng.random((1, cfg["in_chans"], h, w), dtype=np.float32)
                items.append(np.repeat(one, t, axis=0))
            else:
                items.append(rng.random((t, cfg["in_chans"], h, w), dtype=np.float32))
    if cfg["dtype"] == "bf16":
        items = [round_to_bf16(a) for a in items]
    return items


def arrival_trace(n, rate, cv=1.0, seed=0):
    """n request arrival times (seconds, from 0) with i.i.d. Gamma
    inter-arrival gaps of mean 1/rate and coefficient of variation cv
    (cv = 1: Poisson arrivals).  The arrival patterns of the sensitivity
    study (Section 4.5, Table 7) use cv 0.5, 1 and 2."""
    rng = np.random.Generator(np.random.PCG64(seed + 2))
    shape = 1.0 / (cv * cv)
    gaps = rng.gamma(shape, 1.0 / (rate * shape), size=n)
    return np.cumsum(gaps) - gaps[0]

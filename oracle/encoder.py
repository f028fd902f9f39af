"""Plain fp64 CPU reference of the Encode-stage encoder forward pass.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The
product path (the HIP library and its binding) never touches it, and this
module imports nothing from the product package: inputs arrive as numpy
arrays and config dicts.

What it computes.  Encode runs a modality encoder and a lightweight connector
that turn a raw image, clip or audio input into the embedding vectors the LLM
consumes (Section 2.1); the encode worker runs it on micro-batches of up to B
requests (Section 3.2), and each request's embeddings are then shipped on as
one contiguous block (Section 3.3, envelope transfer).  The paper names the
encoders (CLIP ViT-L, a dynamic-resolution ViT, Whisper; Table 3) but does
not spell out their layers, so the layer maths here is the textbook pre-LN
transformer encoder:

* patch embedding = im2col of the pixels followed by a matrix product; the
  audio front end = two kernel-3 1-D convolutions with GELU;
* per layer: x += Wo * Attn(RoPE(LN1(x) Wqkv)),  x += W2 act(W1 LN2(x));
* attention is full (non-causal) within each packed sequence and never
  crosses sequences (block-diagonal over the ``cu_seqlens`` boundaries);
* connector: the 2x2 patch merger (LN, then 4 neighbouring tokens
  concatenated, Linear-GELU-Linear) for merger presets, LN for audio, none for
  the CLS model.

Everything is float64 and written for a reader to check by eye: numpy's
matmul is the only library step; nothing is blocked, fused or reordered.

Pins (tests/test_oracle_pins.py): every part is checked against something
other than itself -- brute-force masked attention, closed forms, torch's
layer norm, attention, convolutions and pre-LN encoder layer, a normal-CDF
table for GELU, RoPE identities, and an explicit spatial gather for the merger.
Parity unpinned: whole-encoder outputs against the paper, which prints no
encoder outputs to compare with.
"""
import math

import numpy as np
from scipy.special import erf as _erf

KIND_VIT_ABS = "vit_abs"
KIND_VIT_CLS_ABS = "vit_cls_abs"
KIND_VIT_ROPE = "vit_rope"
KIND_WHISPER = "whisper"


# ----------------------------------------------------------------------------
# elementwise pieces
# ----------------------------------------------------------------------------

def layer_norm(x, g, b, eps):
    """(x - mean) / sqrt(var + eps) * g + b over the last axis; var is the
    population variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu(x):
    """Exact GELU: x * Phi(x) = x * (1 + erf(x / sqrt 2)) / 2."""
    return x * 0.5 * (1.0 + _erf(x / math.sqrt(2.0)))


def quick_gelu(x):
    """QuickGELU: x * sigmoid(1.702 x)."""
    return x / (1.0 + np.exp(-1.702 * x))


def activation(name):
    return {"gelu": gelu, "quick_gelu": quick_gelu}[name]


def softmax_rows(s):
    m = s.max(axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / e.sum(axis=-1, keepdims=True)


# ----------------------------------------------------------------------------
# packing: raw items -> one padding-free micro-batch
# ----------------------------------------------------------------------------

def token_positions(t, h, w, merge):
    """(ti, hi, wi) of each token of a t x h x w patch grid, in storage order.

    merge == 2: merge-window order -- the four tokens of each 2x2 window are
    consecutive, windows in raster order, so the merger's grouping of 4
    consecutive tokens is the 2x2 spatial neighbourhood.  merge == 1: raster
    order (ti, hi, wi).
    """
    pos = []
    if merge == 2:
        for ti in range(t):
            for hb in range(h // 2):
                for wb in range(w // 2):
                    for dh in range(2):
                        for dw in range(2):
                            pos.append((ti, 2 * hb + dh, 2 * wb + dw))
    else:
        for ti in range(t):
            for hi in range(h):
                for wi in range(w):
                    pos.append((ti, hi, wi))
    return np.array(pos, dtype=np.int64).reshape(-1, 3)


def patch_rows(cfg, item):
    """One item [frames, C, H, W] -> patch vectors in storage order.

    The vector of patch (ti, hi, wi) lists pixel[ti*tp + tau, c, hi*p + dy,
    wi*p + dx] with index ((c*tp + tau)*p + dy)*p + dx, the flatten order of a
    [hidden, C, tp, p, p] convolution weight.
    """
    p, tp = cfg["patch"], cfg["temporal_patch"]
    T, Cc, H, W = item.shape
    t, h, w = T // tp, H // p, W // p
    assert (t * tp, h * p, w * p) == (T, H, W), "item does not tile into patches"
    assert cfg["merge"] == 1 or (h % 2 == 0 and w % 2 == 0), "2x2 merger needs an even patch grid"
    raster = (item.astype(np.float64)
              .reshape(t, tp, Cc, h, p, w, p)
              .transpose(0, 3, 5, 2, 1, 4, 6)       # t, h, w, C, tp, dy, dx
              .reshape(t * h * w, Cc * tp * p * p))
    pos = token_positions(t, h, w, cfg["merge"])
    order = (pos[:, 0] * h + pos[:, 1]) * w + pos[:, 2]
    return raster[order], (t, h, w)


def pack(cfg, items):
    """Concatenate a micro-batch without padding.

    Returns (packed, cu_seqlens, grid_thw).  Vision: packed [N, K] patch rows;
    the CLS model reserves one all-zero row at the start of each sequence for
    its CLS token.  Audio: packed [n, frames, mels] (time-major mel).
    cu_seqlens holds the prefix sums of the per-request token counts.
    """
    if cfg["kind"] == KIND_WHISPER:
        packed = np.stack([np.asarray(m, np.float64).T for m in items])
        L = cfg["n_frames"] // 2
        cu = np.arange(len(items) + 1, dtype=np.int64) * L
        return packed, cu, None
    rows, grids, lens = [], [], []
    for it in items:
        r, g = patch_rows(cfg, it)
        if cfg["kind"] == KIND_VIT_CLS_ABS:
            r = np.concatenate([np.zeros((1, r.shape[1])), r])
        rows.append(r)
        grids.append(g)
        lens.append(r.shape[0])
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    return np.concatenate(rows), cu, np.array(grids, dtype=np.int64)


def sequence_positions(cfg, cu, grid):
    """(t, h, w) of every packed token (the CLS slot gets (0, 0, 0))."""
    out = []
    for r in range(len(cu) - 1):
        t, h, w = (int(v) for v in grid[r])
        pos = token_positions(t, h, w, cfg["merge"])
        if cfg["kind"] == KIND_VIT_CLS_ABS:
            pos = np.concatenate([np.zeros((1, 3), np.int64), pos])
        out.append(pos)
    return np.concatenate(out)


# ----------------------------------------------------------------------------
# embedding
# ----------------------------------------------------------------------------

def conv1d_k3(x, w, b, stride):
    """1-D convolution, kernel 3, zero padding 1 on both sides.

    x [T, Cin] (time-major), w [Cout, Cin*3] flattened in (c, k) order:
    y[t, o] = b[o] + sum_{c,k} w[o, c*3 + k] * x[stride*t + k - 1, c].
    """
    T, cin = x.shape
    cout = w.shape[0]
    tout = (T + 2 - 3) // stride + 1
    wk = w.reshape(cout, cin, 3)
    xp = np.zeros((T + 2, cin))
    xp[1:T + 1] = x
    y = np.tile(b, (tout, 1))
    for k in range(3):
        y = y + xp[k:k + stride * (tout - 1) + 1:stride] @ wk[:, :, k].T
    return y


def sinusoids(length, channels, max_timescale=10000.0):
    """Whisper-style table: [sin | cos] halves, timescales
    exp(-i * ln(max_timescale) / (channels/2 - 1)), i < channels/2."""
    half = channels // 2
    inv = np.exp(-math.log(max_timescale) / (half - 1) * np.arange(half))
    ang = np.arange(length)[:, None] * inv[None, :]
    return np.concatenate([np.sin(ang), np.cos(ang)], axis=1)


def embed(cfg, W, packed, cu, grid):
    """Token embeddings [N, d] of a packed micro-batch (before the layers)."""
    kind = cfg["kind"]
    if kind == KIND_WHISPER:
        xs = []
        for m in packed:
            y = gelu(conv1d_k3(m, W["conv1.w"], W["conv1.b"], 1))
            y = gelu(conv1d_k3(y, W["conv2.w"], W["conv2.b"], 2))
            xs.append(y + sinusoids(y.shape[0], cfg["hidden"]))
        return np.concatenate(xs)
    x = packed @ W["patch.w"].T + W["patch.b"]
    pos = sequence_positions(cfg, cu, grid)
    if kind == KIND_VIT_ABS:
        gw = cfg["pos_grid"][1]
        x = x + W["pos"][pos[:, 1] * gw + pos[:, 2]]
    elif kind == KIND_VIT_CLS_ABS:
        gw = cfg["pos_grid"][1]
        idx = 1 + pos[:, 1] * gw + pos[:, 2]
        idx[cu[:-1]] = 0
        x[cu[:-1]] = W["cls"]
        x = x + W["pos"][idx]
        x = layer_norm(x, W["ln_pre.g"], W["ln_pre.b"], cfg["ln_eps"])
    return x


# ----------------------------------------------------------------------------
# rotary positions
# ----------------------------------------------------------------------------

def rope_angles(pos, sections, theta):
    """Angle of each rotation slot, [N, sum(sections)].

    Slots are split into consecutive sections for the t, h and w axes; slot j
    of an axis with n slots turns by pos_axis * theta**(-j / n).
    """
    cols = []
    for axis, n in enumerate(sections):
        if n == 0:
            continue
        j = np.arange(n, dtype=np.float64)
        cols.append(pos[:, axis:axis + 1].astype(np.float64) * theta ** (-j / n))
    return np.concatenate(cols, axis=1)


def apply_rope(x, ang):
    """Rotate the pairs (k, k + half) of x [N, H, hd] by ang [N, half]."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


# ----------------------------------------------------------------------------
# attention
# ----------------------------------------------------------------------------

def attention_probs(q, k):
    """softmax(q k^T / sqrt(hd)) for one sequence and head."""
    return softmax_rows(q @ k.T / math.sqrt(q.shape[-1]))


def attention(q, k, v, cu):
    """Block-diagonal attention over packed sequences, q/k/v [N, H, hd]."""
    out = np.zeros_like(v)
    for r in range(len(cu) - 1):
        a, b = int(cu[r]), int(cu[r + 1])
        for h in range(q.shape[1]):
            out[a:b, h] = attention_probs(q[a:b, h], k[a:b, h]) @ v[a:b, h]
    return out


# ----------------------------------------------------------------------------
# layers, connector, whole forward
# ----------------------------------------------------------------------------

def encoder_layer(cfg, W, i, x, cu, ang):
    """One pre-LN transformer layer."""
    p = "layers.%d." % i
    d, H, hd = cfg["hidden"], cfg["heads"], cfg["head_dim"]
    eps = cfg["ln_eps"]
    N = x.shape[0]
    a = layer_norm(x, W[p + "ln1.g"], W[p + "ln1.b"], eps)
    qkv = a @ W[p + "qkv.w"].T + W[p + "qkv.b"]
    q = qkv[:, 0 * d:1 * d].reshape(N, H, hd)
    k = qkv[:, 1 * d:2 * d].reshape(N, H, hd)
    v = qkv[:, 2 * d:3 * d].reshape(N, H, hd)
    if ang is not None:
        q, k = apply_rope(q, ang), apply_rope(k, ang)
    o = attention(q, k, v, cu).reshape(N, d)
    x = x + o @ W[p + "o.w"].T + W[p + "o.b"]
    a = layer_norm(x, W[p + "ln2.g"], W[p + "ln2.b"], eps)
    x = x + activation(cfg["act"])(a @ W[p + "fc1.w"].T + W[p + "fc1.b"]) @ W[p + "fc2.w"].T + W[p + "fc2.b"]
    return x


def merger(cfg, W, x):
    """2x2 patch merger: LN, groups of 4 consecutive tokens concatenated to
    4d, then Linear -> GELU -> Linear."""
    d = cfg["hidden"]
    y = layer_norm(x, W["ln_q.g"], W["ln_q.b"], cfg["merger_ln_eps"])
    z = y.reshape(-1, 4 * d)
    return gelu(z @ W["m1.w"].T + W["m1.b"]) @ W["m2.w"].T + W["m2.b"]


def hidden_states(cfg, W, packed, cu, grid, layers=None):
    """Residual stream after ``layers`` layers (default: all)."""
    W = {k: np.asarray(v, np.float64) for k, v in W.items()}
    x = embed(cfg, W, np.asarray(packed, np.float64), cu, grid)
    ang = None
    if cfg["kind"] == KIND_VIT_ROPE:
        ang = rope_angles(sequence_positions(cfg, cu, grid), cfg["rope_sections"], cfg["rope_theta"])
    n = cfg["layers"] if layers is None else layers
    for i in range(n):
        x = encoder_layer(cfg, W, i, x, cu, ang)
    return x


def encode(cfg, W, packed, cu, grid):
    """Whole Encode forward of one micro-batch.

    Returns (out [sum rows, out_dim], cu_out): each request's embeddings as
    contiguous rows in request order, cu_out their prefix sums.
    """
    x = hidden_states(cfg, W, packed, cu, grid)
    W = {k: np.asarray(v, np.float64) for k, v in W.items()}
    if cfg["merge"] == 2:
        out = merger(cfg, W, x)
        cu_out = np.asarray(cu, np.int64) // 4
    elif cfg["kind"] == KIND_WHISPER:
        out = layer_norm(x, W["ln_post.g"], W["ln_post.b"], cfg["ln_eps"])
        cu_out = np.asarray(cu, np.int64)
    else:
        out = x
        cu_out = np.asarray(cu, np.int64)
    return out, cu_out

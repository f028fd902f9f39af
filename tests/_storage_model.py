"""Where the bf16 mode rounds: the fp64 reference with bf16 storage points.

Test infrastructure (a diagnostic beside the fp64 reference, not a second
reference).  The bf16 encoder computes in fp32 but stores its activations in
bf16 between kernels: the LayerNorm outputs that feed a GEMM, the q / k / v
rows (rotary models: q and k once, after the rotary step, where the q | k | v
GEMM's epilogue rotates them; else again after a separate rotary pass), the
softmax probabilities that feed the
P V product, the attention output, the MLP hidden activations, the Whisper
front end's first convolution and the merger's hidden layer.  The residual
stream and the embeddings stay fp32.  ``encode`` below is the reference's
forward pass (the textbook pre-LN encoder of ``oracle/encoder.py``, built
from its own functions) with exactly those values rounded to bf16
(round-to-nearest-even) and everything else in float64.

What it is for.  When attention rows are nearly one-hot (logits of standard
deviation in the tens), a row's output is ill-conditioned in q and k: a
perturbation of one bf16 unit in the last place of a query can move weight
between two keys whose logits nearly tie.  The distance between this model and
the exact reference is then the error that bf16 storage alone implies, before
any kernel arithmetic; a bf16 encoder cannot be expected to land closer to the
exact reference than that.

Pinned in tests/test_storage_model.py: with rounding switched off it equals
the reference's ``encode`` to float64 rounding for every encoder kind.
"""
import math

import numpy as np

from oracle import encoder as O
from paper_2609_31551_amd import synth


def _bf16(a):
    return synth.round_to_bf16(np.asarray(a, np.float32)).astype(np.float64)


def _same(a):
    return a


def _attention(q, k, v, cu, rnd):
    """Block-diagonal attention; the unnormalised probabilities exp(s - max)
    are stored (rnd) before both the P V product and the row sum."""
    out = np.zeros_like(v)
    for r in range(len(cu) - 1):
        a, b = int(cu[r]), int(cu[r + 1])
        for h in range(q.shape[1]):
            s = q[a:b, h] @ k[a:b, h].T / math.sqrt(q.shape[-1])
            p = rnd(np.exp(s - s.max(axis=1, keepdims=True)))
            out[a:b, h] = (p @ v[a:b, h]) / p.sum(axis=1, keepdims=True)
    return out


def _embed(cfg, W, packed, cu, grid, rnd):
    if cfg["kind"] != O.KIND_WHISPER:
        return O.embed(cfg, W, packed, cu, grid)   # GEMM into the fp32 residual stream
    xs = []
    for m in packed:
        y = rnd(O.gelu(O.conv1d_k3(m, W["conv1.w"], W["conv1.b"], 1)))
        y = O.gelu(O.conv1d_k3(y, W["conv2.w"], W["conv2.b"], 2))
        xs.append(y + O.sinusoids(y.shape[0], cfg["hidden"]))
    return np.concatenate(xs)


def rope_in_epilogue(cfg):
    """The library's rule for rotating q and k in the q | k | v GEMM's
    epilogue (bf16 rotary models whose GEMM runs whole 64-wide k-steps)."""
    return cfg["kind"] == O.KIND_VIT_ROPE and cfg["hidden"] % 64 == 0 and cfg["head_dim"] % 8 == 0


def encode(cfg, W, packed, cu, grid, rounding=True):
    """(out, cu_out) like ``oracle.encoder.encode``, with bf16 storage points
    when ``rounding`` is true."""
    rnd = _bf16 if rounding else _same
    W = {k: np.asarray(v, np.float64) for k, v in W.items()}
    x = _embed(cfg, W, np.asarray(packed, np.float64), cu, grid, rnd)
    ang = None
    if cfg["kind"] == O.KIND_VIT_ROPE:
        ang = O.rope_angles(O.sequence_positions(cfg, cu, grid), cfg["rope_sections"], cfg["rope_theta"])
    d, H, hd = cfg["hidden"], cfg["heads"], cfg["head_dim"]
    N = x.shape[0]
    for i in range(cfg["layers"]):
        p = "layers.%d." % i
        a = rnd(O.layer_norm(x, W[p + "ln1.g"], W[p + "ln1.b"], cfg["ln_eps"]))
        qkv = a @ W[p + "qkv.w"].T + W[p + "qkv.b"]
        fused = ang is not None and rope_in_epilogue(cfg)
        if not fused:
            qkv = rnd(qkv)
        q = qkv[:, 0 * d:1 * d].reshape(N, H, hd)
        k = qkv[:, 1 * d:2 * d].reshape(N, H, hd)
        v = qkv[:, 2 * d:3 * d].reshape(N, H, hd)
        if fused:
            v = rnd(v)
        if ang is not None:
            q, k = rnd(O.apply_rope(q, ang)), rnd(O.apply_rope(k, ang))
        o = rnd(_attention(q, k, v, cu, rnd).reshape(N, d))
        x = x + o @ W[p + "o.w"].T + W[p + "o.b"]
        a = rnd(O.layer_norm(x, W[p + "ln2.g"], W[p + "ln2.b"], cfg["ln_eps"]))
        hmid = rnd(O.activation(cfg["act"])(a @ W[p + "fc1.w"].T + W[p + "fc1.b"]))
        x = x + hmid @ W[p + "fc2.w"].T + W[p + "fc2.b"]
    if cfg["merge"] == 2:
        y = rnd(O.layer_norm(x, W["ln_q.g"], W["ln_q.b"], cfg["merger_ln_eps"]))
        z = rnd(O.gelu(y.reshape(-1, 4 * d) @ W["m1.w"].T + W["m1.b"]))
        return z @ W["m2.w"].T + W["m2.b"], np.asarray(cu, np.int64) // 4
    if cfg["kind"] == O.KIND_WHISPER:
        return O.layer_norm(x, W["ln_post.g"], W["ln_post.b"], cfg["ln_eps"]), np.asarray(cu, np.int64)
    return x, np.asarray(cu, np.int64)

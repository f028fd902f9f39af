"""Encoder presets for the Encode stage's modality encoders.

The paper names the encoders only by family (CLIP ViT-L for images, a
dynamic-resolution ViT for video, Whisper for audio; Section 4.1, Table 3)
and runs them as the first stage of the disaggregated pipeline (Section 2.1).
It gives no layer dimensions, so the shapes below are those of the five
workloads this library is built and measured on:

* ``TINY``        -- 2-layer fp32 ViT, 16 tokens per 56x56 image, 2x2 merger.
* ``CLIP_L336``   -- CLIP ViT-L/14 at 336 px: 576 patches + CLS, 24 layers.
* ``QWEN_IMAGE``  -- Qwen2-VL-style variable-resolution ViT, 2D RoPE, merger.
* ``QWEN_VIDEO``  -- the same encoder on 16x448x448 clips, 3D RoPE.
* ``WHISPER_L``   -- Whisper-large-style audio encoder on 128x3000 mel.

Every preset is plain data (a dict of ``eas_config`` fields); it carries no
arithmetic.  ``with_layers`` derives the depth-reduced variants used where
the fp64 reference would otherwise take minutes.
"""

KIND_VIT_ABS = "vit_abs"          # learned absolute positions, no CLS
KIND_VIT_CLS_ABS = "vit_cls_abs"  # CLS token + learned absolute positions + ln_pre
KIND_VIT_ROPE = "vit_rope"        # 2D/3D rotary positions on the patch grid
KIND_WHISPER = "whisper"          # two conv1d layers + sinusoid positions

_BASE = dict(
    in_chans=3, patch=14, temporal_patch=1, merge=1, out_dim=0,
    ln_eps=1e-5, merger_ln_eps=1e-6, rope_theta=10000.0,
    rope_sections=(0, 0, 0), pos_grid=(0, 0), n_mels=0, n_frames=0,
)

TINY = dict(_BASE, name="tiny_vit", kind=KIND_VIT_ABS, dtype="fp32", layers=2,
            hidden=64, heads=4, head_dim=16, mlp=256, act="gelu",
            merge=2, out_dim=128, pos_grid=(4, 4))

CLIP_L336 = dict(_BASE, name="clip_vit_l14_336", kind=KIND_VIT_CLS_ABS, dtype="bf16",
                 layers=24, hidden=1024, heads=16, head_dim=64, mlp=4096,
                 act="quick_gelu", merge=1, out_dim=1024, pos_grid=(24, 24))

QWEN_IMAGE = dict(_BASE, name="qwen2vl_vit_image", kind=KIND_VIT_ROPE, dtype="bf16",
                  layers=32, hidden=1280, heads=16, head_dim=80, mlp=5120,
                  act="quick_gelu", temporal_patch=2, merge=2, out_dim=3584,
                  ln_eps=1e-6, rope_sections=(0, 20, 20))

QWEN_VIDEO = dict(QWEN_IMAGE, name="qwen2vl_vit_video", rope_sections=(8, 16, 16))

WHISPER_L = dict(_BASE, name="whisper_large_enc", kind=KIND_WHISPER, dtype="bf16",
                 layers=32, hidden=1280, heads=20, head_dim=64, mlp=5120, act="gelu",
                 in_chans=1, patch=1, merge=1, out_dim=1280, n_mels=128, n_frames=3000)

PRESETS = {c["name"]: c for c in (TINY, CLIP_L336, QWEN_IMAGE, QWEN_VIDEO, WHISPER_L)}


def with_layers(cfg, layers):
    """Same widths, different depth (used for depth-reduced parity runs)."""
    out = dict(cfg)
    out["layers"] = int(layers)
    out["name"] = "%s_L%d" % (cfg["name"], layers)
    return out


def k_patch(cfg):
    """Length of one packed patch row: C * temporal_patch * patch * patch."""
    if cfg["kind"] == KIND_WHISPER:
        return cfg["n_mels"]
    return cfg["in_chans"] * cfg["temporal_patch"] * cfg["patch"] * cfg["patch"]

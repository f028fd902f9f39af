"""Builds libeas.so (all HIP kernels + the C ABI) in-tree for gfx950 with hipcc."""
import concurrent.futures
import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libeas.so")
BUILD = os.path.join(os.path.dirname(HERE), "_build", "eas")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
         # never emit packed-fp32 VALU ops (v_pk_*_f32)
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


# per-file flags: the attention kernels keep their MFMA accumulators in VGPRs
# (the softmax works on them with VALU ops; AGPRs would need a copy each way),
# and their running maxima are taken without NaN-quieting copies (the scores
# are finite or -inf there, never NaN)
FILE_FLAGS = {"attention_dma.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form", "-fno-honor-nans"]}


# Host-code sanitizers (AddressSanitizer + UndefinedBehaviorSanitizer) for a
# CPU test build: each flag applies to the host pass only, device code is
# built as usual.
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def _compile(src, build_dir=None, extra=()):
    obj = os.path.join(build_dir or BUILD, os.path.basename(src) + ".o")
    cmd = [HIPCC] + FLAGS + FILE_FLAGS.get(os.path.basename(src), []) + list(extra) + ["-x", "hip", "-c", src,
                                                                                         "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stderr or "").splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on %s:\n%s" % (src, err))
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def build(verbose=True, sanitize=False):
    """Builds libeas.so; with sanitize=True a host-sanitized copy instead,
    _build/asan/libeas_asan.so (load it with the ASan runtime preloaded)."""
    build_dir = os.path.join(os.path.dirname(BUILD), "asan") if sanitize else BUILD
    out = os.path.join(build_dir, "libeas_asan.so") if sanitize else OUT
    extra = SANITIZE if sanitize else []
    os.makedirs(build_dir, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip"))) + sorted(glob.glob(os.path.join(CSRC, "*.cpp")))
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda src: _compile(src, build_dir, extra), srcs))
    tmp = out + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC"] + extra + ["-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stderr)
    os.replace(tmp, out)
    if verbose:
        print("built", out)
    return out


if __name__ == "__main__":
    build()

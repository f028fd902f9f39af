// Host side of libeas.so: the C ABI declared in include/eas_encoder.h.
//
// eas_encode_microbatch runs the Encode forward pass (paper Section 2.1) on
// one padding-free micro-batch (Section 3.2) as a fixed sequence of kernel
// launches on the caller's stream:
//   embed (patch GEMM + positions [+ CLS, ln_pre] | conv1d x2 + sinusoid)
//   per layer: LN1 stats -> QKV GEMM (LN prologue) [-> RoPE] -> attention
//              -> O GEMM (+residual) -> LN2 stats -> FC1 GEMM (LN prologue, act)
//              -> FC2 GEMM (+residual)
//   connector: merger (LN stats -> GEMM+GELU with LN prologue -> GEMM) | ln_post | none
// Every per-call shape fact travels to the kernels by value (SeqMeta,
// AttnWork), so a call needs no host-to-device copies and no device sync.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/eas_encoder.h"
#include "common.h"

using namespace eas;

// Workspace of eas_encode_microbatch_noalloc: one array per device, part of
// the library's device code object, so no call allocates.  Host code never
// uses its name except to look up its device address (scratch_base); the
// kernels get that address as an argument, like any workspace pointer.
static __device__ __align__(256) char scratch[EAS_NOALLOC_SCRATCH_BYTES];

namespace {

struct TensorDesc {
  std::string name;
  int64_t offset;
  int ndim;
  int64_t shape[2];
  int64_t numel() const { return ndim == 1 ? shape[0] : shape[0] * shape[1]; }
};

struct Layout {
  std::vector<TensorDesc> t;
  int64_t total = 0;
  int64_t elem = 2;
  void add(const std::string& name, int64_t s0, int64_t s1 = -1) {
    TensorDesc d;
    d.name = name;
    d.ndim = s1 < 0 ? 1 : 2;
    d.shape[0] = s0;
    d.shape[1] = s1 < 0 ? 0 : s1;
    d.offset = total;
    total += (d.numel() * elem + 255) / 256 * 256;
    t.push_back(d);
  }
  int64_t off(const std::string& name) const {
    for (const auto& d : t)
      if (d.name == name) return d.offset;
    return -1;
  }
};

int64_t k_patch(const eas_config& c) {
  if (c.kind == EAS_KIND_WHISPER) return c.n_mels;
  return (int64_t)c.in_chans * c.temporal_patch * c.patch * c.patch;
}

Layout build_layout(const eas_config& c) {
  Layout L;
  L.elem = c.dtype == EAS_BF16 ? 2 : 4;
  const int64_t d = c.hidden, f = c.mlp;
  if (c.kind == EAS_KIND_WHISPER) {
    L.add("conv1.w", d, (int64_t)c.n_mels * 3);
    L.add("conv1.b", d);
    L.add("conv2.w", d, d * 3);
    L.add("conv2.b", d);
  } else {
    L.add("patch.w", d, k_patch(c));
    L.add("patch.b", d);
  }
  const int64_t gh = c.pos_grid[0], gw = c.pos_grid[1];
  if (c.kind == EAS_KIND_VIT_CLS_ABS) {
    L.add("cls", d);
    L.add("pos", 1 + gh * gw, d);
    L.add("ln_pre.g", d);
    L.add("ln_pre.b", d);
  } else if (c.kind == EAS_KIND_VIT_ABS) {
    L.add("pos", gh * gw, d);
  }
  for (int i = 0; i < c.layers; ++i) {
    const std::string p = "layers." + std::to_string(i) + ".";
    L.add(p + "ln1.g", d);
    L.add(p + "ln1.b", d);
    L.add(p + "qkv.w", 3 * d, d);
    L.add(p + "qkv.b", 3 * d);
    L.add(p + "o.w", d, d);
    L.add(p + "o.b", d);
    L.add(p + "ln2.g", d);
    L.add(p + "ln2.b", d);
    L.add(p + "fc1.w", f, d);
    L.add(p + "fc1.b", f);
    L.add(p + "fc2.w", d, f);
    L.add(p + "fc2.b", d);
  }
  if (c.merge == 2) {
    L.add("ln_q.g", d);
    L.add("ln_q.b", d);
    L.add("m1.w", 4 * d, 4 * d);
    L.add("m1.b", 4 * d);
    L.add("m2.w", c.out_dim, 4 * d);
    L.add("m2.b", c.out_dim);
  }
  if (c.kind == EAS_KIND_WHISPER) {
    L.add("ln_post.g", d);
    L.add("ln_post.b", d);
  }
  return L;
}

// Elements per token of the widest activation buffer an encode pass uses as a
// GEMM or attention operand: qkv (3d), the MLP hidden (mlp), the merger input
// (4d), zero-padded patch rows, and the Whisper front end's im2col rows (two
// conv1 input frames of 3 n_mels per token, 3d per conv2 output frame).
int64_t widest_row(const eas_config& c) {
  const int64_t d = c.hidden, kp = k_patch(c);
  int64_t w = std::max<int64_t>({3 * d, (int64_t)c.mlp, 4 * d, (kp + 63) / 64 * 64});
  if (c.kind == EAS_KIND_WHISPER) w = std::max<int64_t>(w, 6 * (int64_t)c.n_mels);
  return w;
}

// Returns "" when the config is usable, else the reason.
std::string check_config(const eas_config& c, eas_status* st) {
  *st = EAS_ERR_INVALID_ARG;
  if (c.kind < EAS_KIND_VIT_ABS || c.kind > EAS_KIND_WHISPER) return "unknown kind";
  if (c.dtype != EAS_FP32 && c.dtype != EAS_BF16) return "dtype must be EAS_FP32 or EAS_BF16";
  if (c.out_dtype != EAS_FP32 && c.out_dtype != EAS_BF16) return "out_dtype must be EAS_FP32 or EAS_BF16";
  if (c.act != EAS_ACT_GELU && c.act != EAS_ACT_QUICKGELU) return "unknown act";
  if (c.layers < 0 || c.hidden <= 0 || c.heads <= 0 || c.head_dim <= 0 || c.mlp <= 0) return "non-positive width";
  if (c.heads * c.head_dim != c.hidden) return "heads * head_dim != hidden";
  if (c.merge != 1 && c.merge != 2) return "merge must be 1 or 2";
  if (c.merge == 2 && c.kind != EAS_KIND_VIT_ABS && c.kind != EAS_KIND_VIT_ROPE) return "merger needs a ViT kind";
  if (c.merge == 2 && c.out_dim <= 0) return "out_dim must be positive with the merger";
  if (c.merge == 1 && c.out_dim != c.hidden) return "out_dim must equal hidden without a merger";
  if (c.max_tokens <= 0 || c.max_tokens > (1L << 30)) return "max_tokens out of range";
  if (c.max_seqs <= 0 || c.max_seqs > EAS_MAX_SEQS) return "max_seqs out of range";
  if (!(c.ln_eps > 0.0f) || !(c.merger_ln_eps > 0.0f)) return "LayerNorm eps must be positive";
  if (c.kind == EAS_KIND_WHISPER) {
    if (c.n_mels <= 0 || c.n_frames <= 0 || c.n_frames % 2) return "n_mels / n_frames invalid";
  } else {
    if (c.in_chans <= 0 || c.patch <= 0 || c.temporal_patch <= 0) return "patch geometry invalid";
  }
  if ((c.kind == EAS_KIND_VIT_ABS || c.kind == EAS_KIND_VIT_CLS_ABS) && (c.pos_grid[0] <= 0 || c.pos_grid[1] <= 0))
    return "pos_grid must be positive";
  if (c.kind == EAS_KIND_VIT_ROPE) {
    if (c.head_dim % 2) return "head_dim must be even for RoPE";
    int s = 0;
    for (int i = 0; i < 3; ++i) {
      if (c.rope_sections[i] < 0) return "negative rope section";
      s += c.rope_sections[i];
    }
    if (s != c.head_dim / 2) return "rope_sections must sum to head_dim / 2";
    if (!(c.rope_theta > 0.0f)) return "rope_theta must be positive";
  }
  *st = EAS_ERR_UNSUPPORTED;
  if (c.hidden % 8 || c.mlp % 8 || (c.merge == 2 && c.out_dim % 8)) return "widths must be multiples of 8";
  if (c.hidden > 2048) return "hidden above 2048 is not built";
  if (c.dtype == EAS_BF16 && c.head_dim != 16 && c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 80 &&
      c.head_dim != 128)
    return "bf16 head_dim must be 16, 32, 64, 80 or 128";
  if (c.dtype == EAS_FP32 && c.head_dim != 16 && c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 80)
    return "fp32 head_dim must be 16, 32, 64 or 80";
  // The bf16 GEMM and attention kernels address each operand with 32-bit byte
  // offsets; every per-token buffer stays below 2^31 elements (4 GiB of bf16).
  if ((double)c.max_tokens * (double)widest_row(c) >= 2147483648.0)
    return "max_tokens too large: the widest per-token buffer would reach 2^31 elements";
  *st = EAS_OK;
  return "";
}

// Token count of a request from its input shape (frames, C, H, W); -1 if invalid.
int64_t request_tokens(const eas_config& c, const int32_t* tchw, int32_t* grid, std::string* why) {
  if (c.kind == EAS_KIND_WHISPER) {
    if (tchw[0] != 1 || tchw[1] != 1 || tchw[2] != c.n_mels || tchw[3] != c.n_frames) {
      *why = "audio items must be (1, 1, n_mels, n_frames)";
      return -1;
    }
    if (grid) grid[0] = 1, grid[1] = 1, grid[2] = c.n_frames / 2;
    return c.n_frames / 2;
  }
  const int T = tchw[0], C = tchw[1], H = tchw[2], W = tchw[3];
  if (C != c.in_chans || T <= 0 || H <= 0 || W <= 0 || T % c.temporal_patch || H % c.patch || W % c.patch) {
    *why = "item does not tile into patches";
    return -1;
  }
  const int t = T / c.temporal_patch, h = H / c.patch, w = W / c.patch;
  if (grid) grid[0] = t, grid[1] = h, grid[2] = w;
  return (int64_t)t * h * w + (c.kind == EAS_KIND_VIT_CLS_ABS ? 1 : 0);
}

std::string check_batch(const eas_config& c, const int32_t* cu, const int32_t* grid, int32_t n, eas_status* st) {
  *st = EAS_ERR_INVALID_ARG;
  if (!cu) return "cu_seqlens is NULL";
  if (!grid && c.kind != EAS_KIND_WHISPER) return "grid_thw is NULL";
  *st = EAS_ERR_CAPACITY;
  if (n < 1 || n > c.max_seqs) return "n_seqs outside 1..max_seqs";
  *st = EAS_ERR_SHAPE;
  if (cu[0] != 0) return "cu_seqlens[0] != 0";
  for (int r = 0; r < n; ++r) {
    if (cu[r + 1] <= cu[r]) return "cu_seqlens not strictly increasing";
    const int64_t L = cu[r + 1] - cu[r];
    if (c.kind == EAS_KIND_WHISPER) {
      if (L != c.n_frames / 2) return "audio sequence length != n_frames / 2";
      continue;
    }
    const int t = grid[3 * r], h = grid[3 * r + 1], w = grid[3 * r + 2];
    if (t <= 0 || h <= 0 || w <= 0) return "grid_thw entries must be positive";
    const int64_t want = (int64_t)t * h * w + (c.kind == EAS_KIND_VIT_CLS_ABS ? 1 : 0);
    if (L != want) return "sequence length does not match grid_thw";
    if (c.merge == 2 && (h % 2 || w % 2)) return "2x2 merger needs even h and w";
    if ((c.kind == EAS_KIND_VIT_ABS || c.kind == EAS_KIND_VIT_CLS_ABS) &&
        (t != 1 || h > c.pos_grid[0] || w > c.pos_grid[1]))
      return "patch grid does not fit the position table";
  }
  *st = EAS_ERR_CAPACITY;
  if (cu[n] > c.max_tokens) return "more tokens than max_tokens";
  *st = EAS_OK;
  return "";
}

struct ProfRec {
  const char* kernel;
  hipEvent_t e0, e1;
  double flops, bytes;
};

}  // namespace

// Per-token activation buffers of one encode pass: the encoder's workspace, or
// a row range of it (row r0 onward), so that two halves of a micro-batch can run
// side by side.  Each buffer holds a fixed number of elements per token, which
// bounds every use of it (the Whisper front end included).
struct Workspace {
  float* x;          // residual stream [tokens, d] fp32
  float2* stats;     // (mean, rstd) per token
  void* qkv;         // [tokens, 3d]
  void* ao;          // [tokens, ao_w]: attention output, Whisper im2col of the mel frames
  void* hbuf;        // [tokens, hw]: MLP hidden, merger input, padded patch rows, conv2 im2col
  void* xn;          // LayerNorm output [tokens, d]
  int4* pos3;        // (t, h, w) per token
  int* tab_idx;      // learned-position row per token
};

struct eas_encoder {
  eas_config cfg;
  Layout layout;
  int device = 0;
  char* ws = nullptr;
  float* x = nullptr;        // residual stream [max_tokens, d] fp32
  float2* stats = nullptr;   // (mean, rstd) per token
  void* qkv = nullptr;       // [max_tokens, 3d]
  void* ao = nullptr;        // attention output [max_tokens, d]
  void* hbuf = nullptr;      // MLP hidden [max_tokens, max(f, 4d, 3d)]
  void* xn = nullptr;        // LayerNorm output [max_tokens, d] (bf16 models)
  int4* pos3 = nullptr;      // (t, h, w) per token
  int* tab_idx = nullptr;    // learned-position row per token
  float* sinus = nullptr;    // [n_frames/2, d] (WHISPER)
  float* inv_freq = nullptr; // [head_dim/2] (VIT_ROPE)
  int* slot_axis = nullptr;  // [head_dim/2]
  int kpad = 0;              // bf16 ViT with a patch row of k_patch % 64 != 0: k_patch rounded up to 64
  void* patch_w = nullptr;   // patch weight [hidden, kpad], zero columns past k_patch (bf16)
  void* qkv_bias = nullptr;  // bf16 rotary ViT: every layer's q | k | v bias, q and k interleaved [layers, 3d]
  int64_t ao_w = 0, hw = 0;  // elements per token of ao and hbuf
  hipStream_t side = nullptr;                          // second half of a split micro-batch
  bool halves = false;                                 // the call in flight runs as two halves
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  hipEvent_t ev_done = nullptr;   // recorded on the caller's stream after each encode call

  Workspace rows_from(int64_t r0) const {
    const int64_t d = cfg.hidden, el = cfg.dtype == EAS_BF16 ? 2 : 4;
    return {x + r0 * d, stats + r0, static_cast<char*>(qkv) + r0 * 3 * d * el, static_cast<char*>(ao) + r0 * ao_w * el,
            static_cast<char*>(hbuf) + r0 * hw * el, static_cast<char*>(xn) + r0 * d * el, pos3 + r0, tab_idx + r0};
  }
  std::string err;
  bool prof = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
};

namespace {

// Bytes of each workspace buffer of an encode pass over up to n tokens, in
// the order bind_workspace lays them out (each 256-byte aligned).
struct WsPlan {
  int64_t sz[12];
  int64_t total = 0;
  int64_t ao_w = 0, hw = 0;   // elements per token of ao and hbuf
  int kpad = 0;
  bool rope = false;          // rotary positions in the q | k | v GEMM's epilogue
};

// bf16 rotary ViTs rotate q and k in the q | k | v GEMM's epilogue when its
// operands meet the DMA kernels' requirements (k a whole number of 64-wide
// steps, head_dim % 8 == 0); the separate rotary pass serves the rest.
bool rope_in_epilogue(const eas_config& c) {
  return c.dtype == EAS_BF16 && c.kind == EAS_KIND_VIT_ROPE && c.layers > 0 && c.hidden % 64 == 0 &&
         c.head_dim % 8 == 0;
}

WsPlan plan_workspace(const eas_config& c, int64_t n) {
  WsPlan w;
  const int64_t d = c.hidden, el = c.dtype == EAS_BF16 ? 2 : 4;
  const int64_t hw = std::max<int64_t>({c.mlp, 4 * d, 3 * d});
  int64_t qkv_rows = n, ao_rows = n;
  if (c.kind == EAS_KIND_WHISPER) {   // front-end im2col and conv1 output reuse qkv / ao
    qkv_rows = std::max<int64_t>(n, (2 * n * d + 3 * d - 1) / (3 * d));
    ao_rows = std::max<int64_t>(n, (2 * n * 3 * c.n_mels + d - 1) / d);
  }
  auto al = [](int64_t b) { return (b + 255) / 256 * 256; };
  const int64_t half = d / c.heads / 2;
  // bf16 ViTs whose patch row is not a whole number of 64-element k-tiles run the
  // embedding GEMM on zero-padded copies (rows in hbuf, weight in patch_w)
  const int64_t kp = k_patch(c), kpad = (kp + 63) / 64 * 64;
  if (c.dtype == EAS_BF16 && c.kind != EAS_KIND_WHISPER && kp % 64 && kpad <= hw) w.kpad = (int)kpad;
  w.rope = rope_in_epilogue(c);
  const int64_t sz[12] = {al(n * d * 4), al(n * 8), al(qkv_rows * 3 * d * el), al(ao_rows * d * el),
                          al(n * hw * el), al(n * 16), al(n * 4),
                          al(c.kind == EAS_KIND_WHISPER ? (int64_t)c.n_frames / 2 * d * 4 : 256),
                          al(half * 8 + 256), al(n * d * el), al(w.kpad ? d * kpad * 2 : 0),
                          al(w.rope ? (int64_t)c.layers * 3 * d * 2 : 0)};
  for (int i = 0; i < 12; ++i) {
    w.sz[i] = sz[i];
    w.total += sz[i];
  }
  w.ao_w = ao_rows * d / n;   // >= d, and >= 6 n_mels for Whisper (two im2col frames per token)
  w.hw = hw;
  return w;
}

void bind_workspace(eas_encoder* e, char* base, const WsPlan& w) {
  char* p = base;
  e->x = (float*)p; p += w.sz[0];
  e->stats = (float2*)p; p += w.sz[1];
  e->qkv = p; p += w.sz[2];
  e->ao = p; p += w.sz[3];
  e->hbuf = p; p += w.sz[4];
  e->pos3 = (int4*)p; p += w.sz[5];
  e->tab_idx = (int*)p; p += w.sz[6];
  e->sinus = (float*)p; p += w.sz[7];
  const int64_t half = e->cfg.hidden / e->cfg.heads / 2;
  e->inv_freq = (float*)p;
  e->slot_axis = (int*)(p + (half * 4 + 255) / 256 * 256);
  p += w.sz[8];
  e->xn = p; p += w.sz[9];
  e->kpad = w.kpad;
  e->patch_w = w.kpad ? p : nullptr;
  p += w.sz[10];
  e->qkv_bias = w.rope ? p : nullptr;
  e->ao_w = w.ao_w;
  e->hw = w.hw;
}

// Whisper's sinusoid table and the rotary slot tables, computed on the device.
hipError_t init_tables(eas_encoder* e, hipStream_t s) {
  const eas_config& c = e->cfg;
  if (c.kind == EAS_KIND_WHISPER) return launch_sinusoid_table(e->sinus, c.n_frames / 2, c.hidden, s);
  if (c.kind == EAS_KIND_VIT_ROPE) return launch_rope_table(e->inv_freq, e->slot_axis, c.rope_sections, c.rope_theta, s);
  return hipSuccess;
}

eas_status fail(eas_encoder* e, eas_status s, const std::string& msg) {
  if (e) e->err = msg;
  return s;
}

hipEvent_t get_event(eas_encoder* e) {
  if (!e->pool.empty()) {
    hipEvent_t ev = e->pool.back();
    e->pool.pop_back();
    return ev;
  }
  hipEvent_t ev = nullptr;
  if (hipEventCreate(&ev) != hipSuccess) return nullptr;
  return ev;
}

// Runs one launch, bracketed by events while profiling is on.
template <class F>
eas_status run(eas_encoder* e, hipStream_t s, double flops, double bytes, F&& launch) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (e->prof) {
    e0 = get_event(e);
    e1 = get_event(e);
    if (e0) (void)hipEventRecord(e0, s);
  }
  const char* kname = "unnamed";
  const hipError_t err = launch(&kname);
  if (e->prof && e0 && e1) {
    (void)hipEventRecord(e1, s);
    e->recs.push_back({kname, e0, e1, flops, bytes});
  }
  if (err != hipSuccess) return fail(e, EAS_ERR_HIP, std::string(kname) + ": " + hipGetErrorString(err));
  return EAS_OK;
}

GemmArgs gemm_args(int M, int N, int K, const void* A, int lda, const void* B, int ldb, void* out, int ldo,
                   int out_f32) {
  GemmArgs g;
  std::memset(&g, 0, sizeof(g));
  g.M = M; g.N = N; g.K = K;
  g.A = A; g.lda = lda;
  g.B = B; g.ldb = ldb;
  g.out = out; g.ldo = ldo; g.out_f32 = out_f32;
  g.ln_group = 1;
  g.pos_period = 1;
  return g;
}

eas_status gemm_launch(eas_encoder* e, const GemmArgs& g, hipStream_t s);

eas_status gemm(eas_encoder* e, const GemmArgs& g, hipStream_t s) {
  if (e->cfg.dtype == EAS_BF16) {
    const int h = gemm_bf16_head_rows(g);
    if (h > 0) {
      const eas_status rc = gemm_launch(e, gemm_rows(g, 0, h), s);
      GemmArgs tail = gemm_rows(g, h, g.M);
      tail.beside = e->halves;
      return rc != EAS_OK ? rc : gemm_launch(e, tail, s);
    }
  }
  return gemm_launch(e, g, s);
}

eas_status gemm_launch(eas_encoder* e, const GemmArgs& g, hipStream_t s) {
  const bool bf = e->cfg.dtype == EAS_BF16;
  const double el = bf ? 2.0 : 4.0;
  const double flops = 2.0 * g.M * g.N * (double)g.K;
  double bytes = (double)g.M * g.K * (g.stats ? 4.0 : el) + (double)g.N * g.K * el + (double)g.M * g.N * (g.out_f32 ? 4.0 : el);
  if (g.resid) bytes += (double)g.M * g.N * 4.0;
  return run(e, s, flops, bytes, [&](const char** kn) {
    return bf ? launch_gemm_bf16(g, s, kn) : launch_gemm_f32(g, s, kn);
  });
}

// LN(x) * W^T: fp32 models fuse the LayerNorm into the GEMM's A loader; bf16
// models write the normalised rows once as bf16 and run the plain GEMM.
// x is [M * group, dim] fp32 viewed as M rows of group * dim.
eas_status ln_gemm(eas_encoder* e, const Workspace& w, GemmArgs g, float eps, int group, hipStream_t s) {
  const int dim = g.ln_dim, rows = g.M * group;
  const float* x = static_cast<const float*>(g.A);
  if (e->cfg.dtype != EAS_BF16) {
    eas_status rc = run(e, s, 0.0, (double)rows * (dim * 4 + 8), [&](const char** kn) {
      *kn = "ln_stats";
      return launch_ln_stats(x, rows, dim, eps, w.stats, s);
    });
    if (rc != EAS_OK) return rc;
    g.stats = w.stats;
    g.ln_group = group;
    return gemm(e, g, s);
  }
  eas_status rc = run(e, s, 0.0, (double)rows * dim * 6, [&](const char** kn) {
    *kn = "ln_apply_bf16";
    return launch_ln_apply(x, rows, dim, eps, g.ln_g, g.ln_b, 1, w.xn, 0, s);
  });
  if (rc != EAS_OK) return rc;
  g.A = w.xn;   // same [M, group * dim] view, now bf16
  g.ln_g = g.ln_b = nullptr;
  return gemm(e, g, s);
}

const char* wptr(const void* weights, const eas_encoder* e, const std::string& name) {
  const int64_t off = e->layout.off(name);
  return off < 0 ? nullptr : static_cast<const char*>(weights) + off;
}

// This call rotates q and k in the q | k | v GEMM's epilogue: the handle has
// the interleaved biases' workspace and the weight rows are 16-byte aligned
// (every layer's are, as layer 0's: tensors sit at 256-byte offsets).
bool rope_fused(const eas_encoder* e, const void* weights) {
  return e->qkv_bias && (uintptr_t)wptr(weights, e, "layers.0.qkv.w") % 16 == 0;
}

}  // namespace

namespace {

// One encode pass over requests cu_seqlens[0 .. n_seqs] (offsets from this
// part's first token) on workspace ws, writing out_embeddings from this part's
// first output row, on stream s.  The caller has checked the batch and prepared
// the padded patch weight.
eas_status encode_part(eas_encoder* enc, const Workspace& ws, const void* packed_in, const int32_t* cu_seqlens,
                       const int32_t* grid_thw, int32_t n_seqs, const void* weights, void* out_embeddings,
                       hipStream_t s) {
  const eas_config& c = enc->cfg;
  const bool bf = c.dtype == EAS_BF16;
  const int out_f32 = c.out_dtype == EAS_FP32;
  const int N = cu_seqlens[n_seqs], d = c.hidden, f = c.mlp, H = c.heads, hd = c.head_dim;
  const int d3 = 3 * d;
  const int64_t el = bf ? 2 : 4;

  SeqMeta meta;
  std::memset(&meta, 0, sizeof(meta));
  meta.n = n_seqs;
  meta.cls = c.kind == EAS_KIND_VIT_CLS_ABS;
  meta.merge = c.merge;
  for (int r = 0; r <= n_seqs; ++r) meta.cu[r] = cu_seqlens[r];
  if (grid_thw)
    for (int r = 0; r < n_seqs; ++r)
      for (int k = 0; k < 3; ++k) meta.thw[r][k] = grid_thw[3 * r + k];

  // attention work list: longest sequences first
  AttnWork work;
  std::memset(&work, 0, sizeof(work));
  work.n = n_seqs;
  for (int r = 0; r <= n_seqs; ++r) work.cu[r] = cu_seqlens[r];
  std::vector<int> ord(n_seqs);
  for (int r = 0; r < n_seqs; ++r) ord[r] = r;
  std::stable_sort(ord.begin(), ord.end(), [&](int a, int b) {
    return cu_seqlens[a + 1] - cu_seqlens[a] > cu_seqlens[b + 1] - cu_seqlens[b];
  });
  // queries per work-list tile of the attention kernel that will run
  AttnArgs probe;
  std::memset(&probe, 0, sizeof(probe));
  probe.qkv = ws.qkv;
  probe.ldqkv = 3 * d;
  probe.hd = hd;
  const int qt = bf && attention_dma_supported(probe, N) ? attention_dma_q_tile(hd, cu_seqlens, n_seqs)
                                                        : attention_q_tile(bf);
  work.qt = qt;
  int tiles = 0;
  double attn_flops = 0.0;
  for (int i = 0; i < n_seqs; ++i) {
    const int r = ord[i];
    const int L = cu_seqlens[r + 1] - cu_seqlens[r];
    work.order[i] = r;
    work.tile_start[i] = tiles;
    tiles += (L + qt - 1) / qt;
    attn_flops += 4.0 * (double)L * L * hd * H;
  }
  work.tile_start[n_seqs] = tiles;

  auto W = [&](const std::string& n) { return wptr(weights, enc, n); };
  eas_status rc = EAS_OK;
#define EAS_TRY(expr)          \
  do {                         \
    rc = (expr);               \
    if (rc != EAS_OK) return rc; \
  } while (0)

  const bool vit = c.kind != EAS_KIND_WHISPER;
  const bool need_pos = vit;
  if (need_pos)
    EAS_TRY(run(enc, s, 0.0, (double)N * 20, [&](const char** kn) {
      *kn = "positions";
      return launch_positions(meta, N, ws.pos3, ws.tab_idx, c.pos_grid[1], s);
    }));

  // ---- embedding ----
  if (vit) {
    const int K = (int)k_patch(c);
    GemmArgs g = gemm_args(N, d, K, packed_in, K, W("patch.w"), K, ws.x, d, 1);
    if (enc->kpad) {   // zero-padded copies: the patch GEMM runs whole 64-wide k-tiles
      const int kp = enc->kpad;
      EAS_TRY(run(enc, s, 0.0, (double)N * (K + kp) * 2, [&](const char** kn) {
        *kn = "pad_cols";
        return launch_pad_cols16(packed_in, N, K, kp, ws.hbuf, s);
      }));
      g = gemm_args(N, d, kp, ws.hbuf, kp, enc->patch_w, kp, ws.x, d, 1);
    }
    g.bias = W("patch.b");
    if (c.kind != EAS_KIND_VIT_ROPE) {
      g.pos = W("pos");
      g.pos_f32 = !bf;
      g.ld_pos = d;
      g.pos_idx = ws.tab_idx;
    }
    EAS_TRY(gemm(enc, g, s));
    if (c.kind == EAS_KIND_VIT_CLS_ABS) {
      EAS_TRY(run(enc, s, 0.0, (double)n_seqs * d * 4, [&](const char** kn) {
        *kn = "cls_insert";
        return launch_cls(meta, ws.x, d, W("cls"), W("pos"), bf, s);
      }));
      EAS_TRY(run(enc, s, 0.0, (double)N * d * 8, [&](const char** kn) {
        *kn = "ln_apply";
        return launch_ln_apply(ws.x, N, d, c.ln_eps, W("ln_pre.g"), W("ln_pre.b"), bf, ws.x, 1, s);
      }));
    }
  } else {
    const int nc = n_seqs, F = c.n_frames, C = c.n_mels;
    // conv1: im2col [nc*F, 3C] (in ao) -> GEMM + GELU -> [nc*F, d] (in qkv)
    EAS_TRY(run(enc, s, 0.0, (double)nc * F * C * 3 * el * 2, [&](const char** kn) {
      *kn = "im2col_k3";
      return launch_im2col_k3(packed_in, F, C, nc, 1, bf, ws.ao, s);
    }));
    GemmArgs g1 = gemm_args(nc * F, d, 3 * C, ws.ao, 3 * C, W("conv1.w"), 3 * C, ws.qkv, d, 0);
    if (!bf) g1.out_f32 = 1;
    g1.bias = W("conv1.b");
    g1.act = ACT_GELU;
    EAS_TRY(gemm(enc, g1, s));
    // conv2 (stride 2): im2col [nc*F/2, 3d] (in hbuf) -> GEMM + GELU + sinusoid -> x
    EAS_TRY(run(enc, s, 0.0, (double)nc * (F / 2) * d * 3 * el * 2, [&](const char** kn) {
      *kn = "im2col_k3";
      return launch_im2col_k3(ws.qkv, F, d, nc, 2, bf, ws.hbuf, s);
    }));
    GemmArgs g2 = gemm_args(N, d, 3 * d, ws.hbuf, 3 * d, W("conv2.w"), 3 * d, ws.x, d, 1);
    g2.bias = W("conv2.b");
    g2.act = ACT_GELU;
    g2.pos = enc->sinus;
    g2.pos_f32 = 1;
    g2.ld_pos = d;
    g2.pos_period = F / 2;
    EAS_TRY(gemm(enc, g2, s));
  }

  // ---- layers ----
  const int act = c.act == EAS_ACT_GELU ? ACT_GELU : ACT_QUICKGELU;
  const bool fuse_rope = rope_fused(enc, weights);
  const int mid_f32 = bf ? 0 : 1;   // qkv / attention / MLP activations: model dtype
  for (int l = 0; l < c.layers; ++l) {
    const std::string p = "layers." + std::to_string(l) + ".";
    GemmArgs gq = gemm_args(N, d3, d, ws.x, d, W(p + "qkv.w"), d, ws.qkv, d3, mid_f32);
    gq.ln_g = W(p + "ln1.g");
    gq.ln_b = W(p + "ln1.b");
    gq.ln_dim = d;
    gq.bias = W(p + "qkv.b");
    if (fuse_rope) {
      gq.bias = static_cast<const char*>(enc->qkv_bias) + (size_t)l * d3 * 2;
      gq.rope_pos = ws.pos3;
      gq.rope_hd = hd;
      gq.rope_hd_inv = rope_hd_inv(hd);
      gq.rope_cols = 2 * d;
      gq.rope_sec0 = c.rope_sections[0];
      gq.rope_sec1 = c.rope_sections[1];
      for (int a = 0; a < 3; ++a)
        gq.rope_c[a] = c.rope_sections[a] > 0 ? (float)(-std::log2((double)c.rope_theta) / c.rope_sections[a]) : 0.0f;
    }
    EAS_TRY(ln_gemm(enc, ws, gq, c.ln_eps, 1, s));
    if (c.kind == EAS_KIND_VIT_ROPE && !fuse_rope)
      EAS_TRY(run(enc, s, 0.0, (double)N * 2 * d * el * 2 + (double)N * 16, [&](const char** kn) {
        *kn = "rope";
        return launch_rope(ws.qkv, d3, N, H, hd, bf, ws.pos3, enc->inv_freq, enc->slot_axis, s);
      }));
    AttnArgs aa;
    aa.qkv = ws.qkv;
    aa.ldqkv = d3;
    aa.out = ws.ao;
    aa.ldo = d;
    aa.heads = H;
    aa.hd = hd;
    aa.scale = (float)(1.0 / std::sqrt((double)hd));
    EAS_TRY(run(enc, s, attn_flops, (double)N * 4 * d * el, [&](const char** kn) {
      return bf ? launch_attention_bf16(aa, work, tiles, N, s, kn) : launch_attention_f32(aa, work, tiles, s, kn);
    }));
    GemmArgs go = gemm_args(N, d, d, ws.ao, d, W(p + "o.w"), d, ws.x, d, 1);
    go.bias = W(p + "o.b");
    go.resid = ws.x;
    go.ldr = d;
    EAS_TRY(gemm(enc, go, s));
    GemmArgs g1 = gemm_args(N, f, d, ws.x, d, W(p + "fc1.w"), d, ws.hbuf, f, mid_f32);
    g1.ln_g = W(p + "ln2.g");
    g1.ln_b = W(p + "ln2.b");
    g1.ln_dim = d;
    g1.bias = W(p + "fc1.b");
    g1.act = act;
    EAS_TRY(ln_gemm(enc, ws, g1, c.ln_eps, 1, s));
    // the CLS model's output is the final residual stream: the last FC2 writes it directly
    const bool direct = c.kind == EAS_KIND_VIT_CLS_ABS && l == c.layers - 1;
    GemmArgs g2 = gemm_args(N, d, f, ws.hbuf, f, W(p + "fc2.w"), f, direct ? out_embeddings : (void*)ws.x, d,
                            direct ? out_f32 : 1);
    g2.bias = W(p + "fc2.b");
    g2.resid = ws.x;
    g2.ldr = d;
    EAS_TRY(gemm(enc, g2, s));
  }

  // ---- connector ----
  if (c.merge == 2) {
    const int G = N / 4, d4 = 4 * d;
    GemmArgs m1 = gemm_args(G, d4, d4, ws.x, d4, W("m1.w"), d4, ws.hbuf, d4, mid_f32);
    m1.ln_g = W("ln_q.g");
    m1.ln_b = W("ln_q.b");
    m1.ln_dim = d;
    m1.bias = W("m1.b");
    m1.act = ACT_GELU;
    EAS_TRY(ln_gemm(enc, ws, m1, c.merger_ln_eps, 4, s));
    GemmArgs m2 = gemm_args(G, c.out_dim, d4, ws.hbuf, d4, W("m2.w"), d4, out_embeddings, c.out_dim, out_f32);
    m2.bias = W("m2.b");
    EAS_TRY(gemm(enc, m2, s));
  } else if (c.kind == EAS_KIND_WHISPER) {
    EAS_TRY(run(enc, s, 0.0, (double)N * d * (4 + (out_f32 ? 4 : 2)), [&](const char** kn) {
      *kn = "ln_apply";
      return launch_ln_apply(ws.x, N, d, c.ln_eps, W("ln_post.g"), W("ln_post.b"), bf, out_embeddings, out_f32, s);
    }));
  } else if (c.layers == 0) {   // CLS model without layers: the embedding is the output
    if (hipMemcpyAsync(out_embeddings, ws.x, (size_t)N * d * 4, hipMemcpyDeviceToDevice, s) != hipSuccess)
      return fail(enc, EAS_ERR_HIP, "hipMemcpyAsync failed");
  }
#undef EAS_TRY
  return EAS_OK;
}

// Large micro-batches are encoded as two halves side by side, requests [0, k)
// and [k, n) split about evenly by tokens: each half's kernels fill the other's
// partial GEMM rounds and overlap its memory-bound steps.  A request's result
// does not depend on the split (every kernel choice gives the same bits).
// The boundary is the first one at or past half the tokens, else the nearest
// within two requests of it whose second-half buffers keep 16-byte alignment
// (CLIP's 588-element patch rows need an even token offset).  Returns k, or 0
// for one pass: per-kernel profiling (one stream of events), small batches,
// and no aligned boundary near the middle.  From 8192 tokens: against 16384,
// CLIP x16 +5.9%, x24 +3.5%, Qwen-style images x4 +1.3%, Whisper x6 +1.0%,
// Whisper x8 -0.8% (same-box A/B); below it the halves lose (CLIP x4 -4%,
// Whisper x4 -7% at a 1024-token threshold).
constexpr int kSplitTokens = 8192;
int split_point(const eas_encoder* e, const int32_t* cu, int n, int64_t* in_off, int64_t* out_off) {
  const eas_config& c = e->cfg;
  if (e->prof || !e->side || n < 2 || cu[n] < kSplitTokens) return 0;
  int k0 = 1;
  while (k0 < n - 1 && 2 * (int64_t)cu[k0] < cu[n]) ++k0;
  const int64_t el = c.dtype == EAS_BF16 ? 2 : 4, oel = c.out_dtype == EAS_FP32 ? 4 : 2;
  for (int k : {k0, k0 - 1, k0 + 1, k0 - 2, k0 + 2}) {
    if (k < 1 || k > n - 1) continue;
    const int64_t r0 = cu[k];
    const int64_t in = c.kind == EAS_KIND_WHISPER ? (int64_t)k * c.n_mels * c.n_frames * el : r0 * k_patch(c) * el;
    const int64_t out = (c.merge == 2 ? r0 / 4 : r0) * c.out_dim * oel;
    const int64_t offs[] = {in, out, r0 * c.hidden * 4, r0 * 3 * c.hidden * el, r0 * e->ao_w * el,
                            r0 * e->hw * el, r0 * c.hidden * el};
    bool ok = true;
    for (int64_t o : offs) ok = ok && o % 16 == 0;
    if (ok) {
      *in_off = in;
      *out_off = out;
      return k;
    }
  }
  return 0;
}

// The Encode pass of one checked micro-batch on handle enc (a created
// handle, or a view over the scratch array), on stream s.
eas_status encode_call(eas_encoder* enc, const void* packed_in, const int32_t* cu_seqlens, const int32_t* grid_thw,
                       int32_t n_seqs, const void* weights, void* out_embeddings, int32_t* cu_out, hipStream_t s) {
  const eas_config& c = enc->cfg;
  if (c.kind == EAS_KIND_VIT_CLS_ABS && c.layers == 0 && c.out_dtype != EAS_FP32)
    return fail(enc, EAS_ERR_UNSUPPORTED, "zero-layer CLS model needs fp32 output");
  eas_status rc = EAS_OK;
  if (enc->kpad) {   // the zero-padded patch weight, shared by both halves of a split call
    const int K = (int)k_patch(c), kp = enc->kpad, d = c.hidden;
    rc = run(enc, s, 0.0, (double)d * (K + kp) * 2, [&](const char** kn) {
      *kn = "pad_cols";
      return launch_pad_cols16(wptr(weights, enc, "patch.w"), d, K, kp, enc->patch_w, s);
    });
    if (rc != EAS_OK) return rc;
  }
  if (rope_fused(enc, weights)) {   // the interleaved q | k | v biases of every layer, shared likewise
    const int d = c.hidden;
    const int64_t o0 = enc->layout.off("layers.0.qkv.b");
    const long stride = c.layers > 1 ? (long)((enc->layout.off("layers.1.qkv.b") - o0) / 2) : 0;
    rc = run(enc, s, 0.0, (double)c.layers * 3 * d * 4, [&](const char** kn) {
      *kn = "rope_bias";
      return launch_rope_bias(static_cast<const char*>(weights) + o0, stride, c.layers, 2 * d, c.head_dim,
                              enc->qkv_bias, s);
    });
    if (rc != EAS_OK) return rc;
  }
  int64_t in_off = 0, out_off = 0;
  const int k = split_point(enc, cu_seqlens, n_seqs, &in_off, &out_off);
  if (k == 0) {
    rc = encode_part(enc, enc->rows_from(0), packed_in, cu_seqlens, grid_thw, n_seqs, weights, out_embeddings, s);
  } else {
    // requests [0, k) on the caller's stream and [k, n) on the encoder's second
    // stream, forked from the caller's stream and joined back into it
    std::vector<int32_t> cub(n_seqs - k + 1);
    for (int r = 0; r <= n_seqs - k; ++r) cub[r] = cu_seqlens[k + r] - cu_seqlens[k];
    if (hipEventRecord(enc->ev_fork, s) != hipSuccess || hipStreamWaitEvent(enc->side, enc->ev_fork, 0) != hipSuccess)
      return fail(enc, EAS_ERR_HIP, "stream fork failed");
    enc->halves = true;
    rc = encode_part(enc, enc->rows_from(0), packed_in, cu_seqlens, grid_thw, k, weights, out_embeddings, s);
    if (rc == EAS_OK)
      rc = encode_part(enc, enc->rows_from(cu_seqlens[k]), static_cast<const char*>(packed_in) + in_off, cub.data(),
                       grid_thw ? grid_thw + 3 * k : nullptr, n_seqs - k, weights,
                       static_cast<char*>(out_embeddings) + out_off, enc->side);
    enc->halves = false;
    // joined even after an error: the caller's stream never runs ahead of the side stream
    const bool joined = hipEventRecord(enc->ev_join, enc->side) == hipSuccess &&
                        hipStreamWaitEvent(s, enc->ev_join, 0) == hipSuccess;
    if (rc == EAS_OK && !joined) rc = fail(enc, EAS_ERR_HIP, "stream join failed");
  }
  if (enc->ev_done && hipEventRecord(enc->ev_done, s) != hipSuccess && rc == EAS_OK)
    rc = fail(enc, EAS_ERR_HIP, "event record failed");
  if (rc != EAS_OK) return rc;
  if (cu_out) {
    for (int r = 0; r <= n_seqs; ++r) cu_out[r] = c.merge == 2 ? cu_seqlens[r] / 4 : cu_seqlens[r];
  }
  enc->err.clear();
  return EAS_OK;
}

// Device address of this device's scratch array, looked up once per device
// (with that device current) and kept; NULL if the lookup fails.
char* scratch_base(int dev) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static char* base[kMaxDevices] = {};
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (!base[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
    base[dev] = static_cast<char*>(p);
  }
  return base[dev];
}

}  // namespace

extern "C" {

const char* eas_status_string(eas_status s) {
  switch (s) {
    case EAS_OK: return "ok";
    case EAS_ERR_INVALID_ARG: return "invalid argument";
    case EAS_ERR_SHAPE: return "shape error";
    case EAS_ERR_CAPACITY: return "capacity exceeded";
    case EAS_ERR_UNSUPPORTED: return "unsupported configuration";
    case EAS_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* eas_last_error(const eas_encoder* enc) { return enc ? enc->err.c_str() : ""; }

eas_status eas_weights_layout(const eas_config* cfg, eas_tensor_desc* descs, int32_t capacity, int32_t* n_descs,
                              int64_t* total_bytes) {
  if (!cfg || !n_descs) return EAS_ERR_INVALID_ARG;
  eas_status st;
  if (!check_config(*cfg, &st).empty()) return st;
  const Layout L = build_layout(*cfg);
  *n_descs = (int32_t)L.t.size();
  if (total_bytes) *total_bytes = L.total;
  if (!descs) return EAS_OK;
  if (capacity < (int32_t)L.t.size()) return EAS_ERR_CAPACITY;
  for (size_t i = 0; i < L.t.size(); ++i) {
    std::memset(&descs[i], 0, sizeof(eas_tensor_desc));
    std::snprintf(descs[i].name, sizeof(descs[i].name), "%s", L.t[i].name.c_str());
    descs[i].offset_bytes = L.t[i].offset;
    descs[i].ndim = L.t[i].ndim;
    descs[i].shape[0] = L.t[i].shape[0];
    descs[i].shape[1] = L.t[i].shape[1];
  }
  return EAS_OK;
}

eas_status eas_microbatch_shape(const eas_config* cfg, int32_t n_req, const int32_t* tchw, int32_t* cu_seqlens,
                                int32_t* grid_thw, int64_t* packed_elems, int64_t* out_rows) {
  if (!cfg || !tchw || !cu_seqlens) return EAS_ERR_INVALID_ARG;
  eas_status st;
  if (!check_config(*cfg, &st).empty()) return st;
  if (n_req < 1 || n_req > cfg->max_seqs) return EAS_ERR_CAPACITY;
  std::string why;
  int64_t tot = 0;
  cu_seqlens[0] = 0;
  for (int r = 0; r < n_req; ++r) {
    int32_t g[3];
    const int64_t L = request_tokens(*cfg, tchw + 4 * r, g, &why);
    if (L < 0) return EAS_ERR_SHAPE;
    if (cfg->merge == 2 && (g[1] % 2 || g[2] % 2)) return EAS_ERR_SHAPE;
    tot += L;
    if (tot > cfg->max_tokens) return EAS_ERR_CAPACITY;
    cu_seqlens[r + 1] = (int32_t)tot;
    if (grid_thw) std::memcpy(grid_thw + 3 * r, g, sizeof(g));
  }
  if (packed_elems) *packed_elems = cfg->kind == EAS_KIND_WHISPER ? (int64_t)n_req * cfg->n_mels * cfg->n_frames
                                                                   : tot * k_patch(*cfg);
  if (out_rows) *out_rows = cfg->merge == 2 ? tot / 4 : tot;
  return EAS_OK;
}

eas_status eas_validate_microbatch(const eas_config* cfg, const int32_t* cu_seqlens, const int32_t* grid_thw,
                                   int32_t n_seqs) {
  if (!cfg) return EAS_ERR_INVALID_ARG;
  eas_status st;
  if (!check_config(*cfg, &st).empty()) return st;
  check_batch(*cfg, cu_seqlens, grid_thw, n_seqs, &st);
  return st;
}

eas_status eas_encoder_create(const eas_config* cfg, eas_encoder** out) {
  if (!cfg || !out) return EAS_ERR_INVALID_ARG;
  *out = nullptr;
  eas_status st;
  const std::string why = check_config(*cfg, &st);
  if (!why.empty()) return st;
  eas_encoder* e = new (std::nothrow) eas_encoder();
  if (!e) return EAS_ERR_HIP;
  e->cfg = *cfg;
  e->layout = build_layout(*cfg);
  if (hipGetDevice(&e->device) != hipSuccess) {
    delete e;
    return EAS_ERR_HIP;
  }
  const WsPlan plan = plan_workspace(*cfg, cfg->max_tokens);
  if (hipMalloc(&e->ws, plan.total) != hipSuccess) {
    delete e;
    return EAS_ERR_HIP;
  }
  bind_workspace(e, e->ws, plan);
  const eas_config& c = *cfg;
  // the position tables, once, on the null stream
  hipError_t herr = init_tables(e, nullptr);
  if (herr == hipSuccess) herr = hipStreamSynchronize(nullptr);
  // second stream and fork / join events for split micro-batches (default
  // priority); without them every call runs as one pass
  if (herr == hipSuccess && c.max_seqs >= 2) {
    if (hipStreamCreateWithFlags(&e->side, hipStreamNonBlocking) != hipSuccess) e->side = nullptr;
    if (e->side && (hipEventCreateWithFlags(&e->ev_fork, hipEventDisableTiming) != hipSuccess ||
                    hipEventCreateWithFlags(&e->ev_join, hipEventDisableTiming) != hipSuccess)) {
      if (e->ev_fork) (void)hipEventDestroy(e->ev_fork);
      (void)hipStreamDestroy(e->side);
      e->side = nullptr;
      e->ev_fork = nullptr;
    }
  }
  if (herr == hipSuccess) herr = hipEventCreateWithFlags(&e->ev_done, hipEventDisableTiming);
  if (herr != hipSuccess) {
    if (e->side) {
      (void)hipEventDestroy(e->ev_fork);
      (void)hipEventDestroy(e->ev_join);
      (void)hipStreamDestroy(e->side);
    }
    (void)hipFree(e->ws);
    delete e;
    return EAS_ERR_HIP;
  }
  *out = e;
  return EAS_OK;
}

void eas_encoder_destroy(eas_encoder* enc) {
  if (!enc) return;
  // only the handle's own work: the last encode call ends with ev_done on the
  // caller's stream (its second half, if any, joined that stream before it;
  // earlier calls were ordered before it, as calls on one handle must be), and
  // the side stream is the handle's own
  if (enc->ev_done) (void)hipEventSynchronize(enc->ev_done);
  if (enc->side) (void)hipStreamSynchronize(enc->side);
  for (auto& r : enc->recs) {
    (void)hipEventDestroy(r.e0);
    (void)hipEventDestroy(r.e1);
  }
  for (auto ev : enc->pool) (void)hipEventDestroy(ev);
  if (enc->ev_done) (void)hipEventDestroy(enc->ev_done);
  if (enc->side) {
    (void)hipEventDestroy(enc->ev_fork);
    (void)hipEventDestroy(enc->ev_join);
    (void)hipStreamDestroy(enc->side);
  }
  (void)hipFree(enc->ws);
  delete enc;
}

eas_status eas_profile_enable(eas_encoder* enc, int32_t enable) {
  if (!enc) return EAS_ERR_INVALID_ARG;
  enc->prof = enable != 0;
  return EAS_OK;
}

eas_status eas_profile_read(eas_encoder* enc, eas_kernel_stat* stats, int32_t capacity, int32_t* n_stats) {
  if (!enc || !n_stats) return EAS_ERR_INVALID_ARG;
  std::vector<eas_kernel_stat> agg;
  for (auto& r : enc->recs) {
    if (hipEventSynchronize(r.e1) != hipSuccess) return fail(enc, EAS_ERR_HIP, "hipEventSynchronize failed");
    float ms = 0.0f;
    (void)hipEventElapsedTime(&ms, r.e0, r.e1);
    eas_kernel_stat* k = nullptr;
    for (auto& a : agg)
      if (std::strcmp(a.kernel, r.kernel) == 0) k = &a;
    if (!k) {
      agg.push_back(eas_kernel_stat());
      k = &agg.back();
      std::memset(k, 0, sizeof(*k));
      std::snprintf(k->kernel, sizeof(k->kernel), "%s", r.kernel);
    }
    k->launches += 1;
    k->total_ms += ms;
    k->flops += r.flops;
    k->bytes += r.bytes;
  }
  *n_stats = (int32_t)agg.size();
  if (!stats) return EAS_OK;
  for (auto& r : enc->recs) {
    enc->pool.push_back(r.e0);
    enc->pool.push_back(r.e1);
  }
  enc->recs.clear();
  for (int32_t i = 0; i < std::min<int32_t>(capacity, (int32_t)agg.size()); ++i) stats[i] = agg[i];
  return capacity < (int32_t)agg.size() ? EAS_ERR_CAPACITY : EAS_OK;
}

eas_status eas_pack_microbatch(eas_encoder* enc, int32_t n_req, const float* const* items, const int32_t* tchw,
                               void* packed, int32_t* cu_seqlens, int32_t* grid_thw, void* stream) {
  if (!enc || !items || !tchw || !packed || !cu_seqlens) return fail(enc, EAS_ERR_INVALID_ARG, "NULL argument");
  const eas_config& c = enc->cfg;
  int32_t cu[EAS_MAX_SEQS + 1], grid[EAS_MAX_SEQS * 3];
  int64_t elems = 0;
  if (n_req < 1 || n_req > c.max_seqs) return fail(enc, EAS_ERR_CAPACITY, "n_req outside 1..max_seqs");
  const eas_status st = eas_microbatch_shape(&c, n_req, tchw, cu, grid, &elems, nullptr);
  if (st != EAS_OK) return fail(enc, st, "item shapes rejected");
  for (int r = 0; r < n_req; ++r)
    if (!items[r]) return fail(enc, EAS_ERR_INVALID_ARG, "NULL item pointer");
  PackArgs p;
  std::memset(&p, 0, sizeof(p));
  p.n = n_req;
  for (int r = 0; r <= n_req; ++r) p.cu[r] = cu[r];
  for (int r = 0; r < n_req; ++r) {
    for (int k = 0; k < 4; ++k) p.tchw[r][k] = tchw[4 * r + k];
    p.src[r] = items[r];
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int bf = c.dtype == EAS_BF16;
  const eas_status rs = run(enc, s, 0.0, (double)elems * (4 + (bf ? 2 : 4)), [&](const char** kn) {
    if (c.kind == EAS_KIND_WHISPER) {
      *kn = "pack_audio";
      return launch_pack_audio(p, c.n_mels, c.n_frames, bf, packed, s);
    }
    *kn = "pack_vision";
    return launch_pack_vision(p, c.kind == EAS_KIND_VIT_CLS_ABS, c.merge, c.patch, c.temporal_patch,
                              (int)k_patch(c), bf, packed, elems, s);
  });
  if (rs != EAS_OK) return rs;
  std::memcpy(cu_seqlens, cu, sizeof(int32_t) * (n_req + 1));
  if (grid_thw) std::memcpy(grid_thw, grid, sizeof(int32_t) * 3 * n_req);
  return EAS_OK;
}

eas_status eas_encode_microbatch(eas_encoder* enc, const void* packed_in, const int32_t* cu_seqlens,
                                 const int32_t* grid_thw, int32_t n_seqs, const void* weights, void* out_embeddings,
                                 int32_t* cu_out, void* stream) {
  if (!enc) return EAS_ERR_INVALID_ARG;
  if (!packed_in || !weights || !out_embeddings) return fail(enc, EAS_ERR_INVALID_ARG, "NULL device pointer");
  eas_status st;
  const std::string why = check_batch(enc->cfg, cu_seqlens, grid_thw, n_seqs, &st);
  if (st != EAS_OK) return fail(enc, st, why);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev != enc->device)
    return fail(enc, EAS_ERR_INVALID_ARG, "current device differs from the handle's device");
  return encode_call(enc, packed_in, cu_seqlens, grid_thw, n_seqs, weights, out_embeddings, cu_out,
                     static_cast<hipStream_t>(stream));
}

eas_status eas_encode_microbatch_noalloc(const eas_config* cfg, const void* packed_in, const int32_t* cu_seqlens,
                                         const int32_t* grid_thw, int32_t n_seqs, const void* weights,
                                         void* out_embeddings, int32_t* cu_out, void* stream) {
  if (!cfg || !packed_in || !weights || !out_embeddings) return EAS_ERR_INVALID_ARG;
  eas_status st;
  if (!check_config(*cfg, &st).empty()) return st;
  check_batch(*cfg, cu_seqlens, grid_thw, n_seqs, &st);
  if (st != EAS_OK) return st;
  const WsPlan plan = plan_workspace(*cfg, cu_seqlens[n_seqs]);
  if (plan.total > (int64_t)EAS_NOALLOC_SCRATCH_BYTES) return EAS_ERR_CAPACITY;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return EAS_ERR_HIP;
  char* base = scratch_base(dev);
  if (!base) return EAS_ERR_HIP;
  // a handle on the host stack over this device's scratch array: no second
  // stream (the micro-batch runs as one pass), no profiling, no events
  eas_encoder view;
  view.cfg = *cfg;
  view.layout = build_layout(*cfg);
  view.device = dev;
  bind_workspace(&view, base, plan);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (init_tables(&view, s) != hipSuccess) return EAS_ERR_HIP;
  return encode_call(&view, packed_in, cu_seqlens, grid_thw, n_seqs, weights, out_embeddings, cu_out, s);
}

}  // extern "C"

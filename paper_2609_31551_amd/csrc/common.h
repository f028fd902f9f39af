// Shared device types, small helpers and the launcher declarations of the
// Encode-stage encoder kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

namespace eas {

constexpr int kMaxSeqs = 64;

// Per-micro-batch sequence metadata, passed to kernels by value.
struct SeqMeta {
  int n;                    // sequences
  int cls;                  // 1 if every sequence starts with a CLS token
  int merge;                // 1 or 2
  int cu[kMaxSeqs + 1];     // token prefix sums
  int thw[kMaxSeqs][3];     // patch grid per sequence
};

// Attention work list: q-tiles of all sequences, longest sequence first.
struct AttnWork {
  int n;                    // sequences
  int cu[kMaxSeqs + 1];
  int order[kMaxSeqs];      // order[i] = sequence handled by the i-th tile group
  int tile_start[kMaxSeqs + 1];  // prefix sums of q-tiles over `order`
  int qt;                   // queries per q-tile
};

enum Act { ACT_NONE = 0, ACT_GELU = 1, ACT_QUICKGELU = 2 };

// GELU(v) = v Phi(v) = 0.5 v (1 + erf(v / sqrt 2)) with erf by Abramowitz &
// Stegun, Handbook of Mathematical Functions, formula 7.1.28:
// erf(x) = 1 - 1 / (1 + a1 x + ... + a6 x^6)^16 for x >= 0, |error| <= 3e-7.
// With P(|v|) = that polynomial at |v| / sqrt 2 (the scale folded into the
// coefficients), GELU(v) = max(v, 0) - 0.5 |v| / P^16 for either sign of v:
// branch-free, one reciprocal and no exponential, in the GEMM epilogues where
// it runs on every output element.  P^16 overflowing to inf for |v| > ~25
// gives the exact limits (v, or -0).
__device__ __forceinline__ float gelu_erf(float v) {
  const float av = fabsf(v);
  float p = fmaf(fmaf(fmaf(fmaf(fmaf(5.38297490e-06f, av, 4.88906371e-05f), av, 3.80035744e-05f), av,
                           3.27762635e-03f), av, 2.11410057e-02f), av, 4.98673469e-02f);
  p = fmaf(p, av, 1.0f);
  p *= p;
  p *= p;
  p *= p;
  p *= p;
  return fmaxf(v, 0.0f) - 0.5f * av * __builtin_amdgcn_rcpf(p);
}
// x sigmoid(1.702 x) = x / (1 + 2^(-1.702 log2(e) x)): one multiply into the
// hardware exponential, and the hardware reciprocal instead of a full-precision divide
__device__ __forceinline__ float quick_gelu(float v) {
  return v * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(v * -2.45546696f));
}
__device__ __forceinline__ float apply_act(int act, float v) {
  if (act == ACT_GELU) return gelu_erf(v);
  if (act == ACT_QUICKGELU) return quick_gelu(v);
  return v;
}

template <class T> __device__ __forceinline__ float to_f(T v) { return (float)v; }
template <class T> __device__ __forceinline__ T from_f(float v) { return (T)v; }

// Row r's sequence: largest s with cu[s] <= r.
__device__ __forceinline__ int find_seq(const int* cu, int n, int r) {
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (cu[mid] <= r) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Fused GEMM epilogue / prologue description:
//   out[m, n] = act(sum_k A'[m, k] * B[n, k] + bias[n]) + pos[idx(m), n] + resid[m, n]
// where A' is A itself, or LayerNorm(A) when `stats` is set:
//   A'[m, k] = (A[m, k] - mu[t]) * rstd[t] * g[k % ln_dim] + b[k % ln_dim],
//   t = m * ln_group + k / ln_dim   (ln_group = 4 views 4 tokens as one row).
struct GemmArgs {
  int M, N, K;
  const void* A; int lda;          // [M, lda]: model dtype, or fp32 when stats != null
  const void* B; int ldb;          // [N, ldb] model dtype
  const float2* stats;             // per token (mean, rstd) or null
  const void* ln_g; const void* ln_b; int ln_dim; int ln_group;
  const void* bias;                // [N] model dtype or null
  int act;
  const void* pos; int pos_f32; int ld_pos;   // position table (model dtype or fp32)
  const int* pos_idx; int pos_period;         // table row: pos_idx[m] or m % pos_period
  const float* resid; int ldr;                // fp32 residual (may alias out)
  void* out; int ldo; int out_f32;
  int beside;                      // the rows a half leaves after whole rounds of 256 x 256 tiles,
                                   // launched while the other half's kernels run on another stream
  // Rotary positions applied in the epilogue of the bf16 q | k | v projection
  // (rope_pos set): output columns [0, rope_cols) are the q and k heads, rope_hd
  // columns each, in interleaved order -- column 2i of a head holds its x_i and
  // column 2i + 1 its x_{i + rope_hd/2} -- so each rotated pair sits in adjacent
  // columns of one lane.  Their weight rows are read from the natural order
  // (rope_src_row) and the bias is passed already interleaved; q . k is the
  // same in either order since q and k share it.  Slots [0, rope_sec0) turn
  // with the t position, the next rope_sec1 with h, the rest with w; rope_c[a]
  // = -log2(theta) / (slots of axis a).
  const int4* rope_pos;            // (t, h, w) per output row, or null
  int rope_hd, rope_cols, rope_sec0, rope_sec1;
  unsigned rope_hd_inv;            // ceil(2^32 / rope_hd): n / rope_hd = umulhi(n, rope_hd_inv) for n < 2^16
  float rope_c[3];
};

// Column n's offset within its head (n < 2^16, hd <= 128: the product's error
// n * (ceil(2^32/hd) - 2^32/hd) / 2^32 < 2^-16 stays below the 1/hd gap to the
// next integer, so the quotient is exact).
__device__ __forceinline__ int rope_in_head(int n, int hd, unsigned hd_inv) {
  return n - (int)__umulhi((unsigned)n, hd_inv) * hd;
}
// Weight row of output column n of an interleaved rotary projection.
__device__ __forceinline__ int rope_src_row(int n, int hd, unsigned hd_inv, int cols) {
  if (n >= cols) return n;
  const int c = rope_in_head(n, hd, hd_inv);
  return n - c + (c >> 1) + (c & 1) * (hd >> 1);
}
// Turns (angle / 2 pi) of rotation slot i at position (pt, ph, pw):
// pos_axis * theta^(-j / n_axis) / (2 pi).  Components by value: selecting
// among the fields of a struct in memory would become an indexed load.
__device__ __forceinline__ float rope_turns(const GemmArgs& a, int i, int pt, int ph, int pw) {
  const bool ht = i < a.rope_sec0, hh = !ht && i < a.rope_sec0 + a.rope_sec1;
  const int j = ht ? i : (hh ? i - a.rope_sec0 : i - a.rope_sec0 - a.rope_sec1);
  const float c = ht ? a.rope_c[0] : (hh ? a.rope_c[1] : a.rope_c[2]);
  const int pos = ht ? pt : (hh ? ph : pw);
  return (float)pos * __builtin_amdgcn_exp2f(fmaf((float)j, c, -2.65149613f));   // 2^(j c - log2(2 pi))
}
// (x, y) = (x_i, x_{i+half}) rotated by `turns`: x cos - y sin, y cos + x sin.  The
// hardware sine and cosine take turns; the fraction (exact) keeps them in range.
__device__ __forceinline__ void rope_rotate(float& x, float& y, float turns) {
  const float t = __builtin_amdgcn_fractf(turns);
  const float cs = __builtin_amdgcn_cosf(t), sn = __builtin_amdgcn_sinf(t);
  const float xr = fmaf(x, cs, -(y * sn));
  y = fmaf(y, cs, x * sn);
  x = xr;
}

// ---- launchers (each returns hipGetLastError() of its launch) --------------
hipError_t launch_gemm_bf16(const GemmArgs& a, hipStream_t s, const char** kname);
inline unsigned rope_hd_inv(int hd) { return (unsigned)((0x100000000ull + (unsigned)hd - 1) / (unsigned)hd); }
// Whether launch_gemm_bf16 runs these arguments with the rotary epilogue (the
// DMA kernels' operand and epilogue requirements, bf16 output, head_dim % 8 == 0).
bool gemm_bf16_rope_ok(const GemmArgs& a);
// Rows [0, h) of a bf16 GEMM whose last round of 256 x 256 tiles would run
// mostly empty: launched as whole rounds, rows [h, M) as a second launch with
// a smaller tile.  0 when one launch is as fast.
int gemm_bf16_head_rows(const GemmArgs& a);
// The same GEMM restricted to output rows [m0, m1) (pointers and row-indexed
// epilogue streams shifted; a period-indexed position table needs
// m0 % pos_period == 0).
GemmArgs gemm_rows(const GemmArgs& a, int m0, int m1);
hipError_t launch_gemm_bf16_staged(const GemmArgs& a, hipStream_t s, const char** kname);
hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s, const char** kname);

struct AttnArgs {
  const void* qkv; int ldqkv;      // [N, ldqkv]: q | k | v blocks of width heads*hd
  void* out; int ldo;              // [N, ldo]
  int heads, hd;
  float scale;                     // 1 / sqrt(hd)
};
hipError_t launch_attention_bf16(const AttnArgs& a, const AttnWork& w, int total_tiles, int N, hipStream_t s,
                                 const char** kname);
// DMA-fed kernel for head_dim 64 / 80, and its queries per work-list tile for
// the sequences of a micro-batch (cu: n + 1 prefix sums)
bool attention_dma_supported(const AttnArgs& a, int N);
int attention_dma_q_tile(int hd, const int* cu, int n);
hipError_t launch_attention_bf16_dma(const AttnArgs& a, const AttnWork& w, int total_tiles, hipStream_t s,
                                     const char** kname);
hipError_t launch_attention_f32(const AttnArgs& a, const AttnWork& w, int total_tiles, hipStream_t s,
                                const char** kname);
int attention_q_tile(int dtype_bf16);

hipError_t launch_positions(const SeqMeta& m, int N, int4* pos3, int* tab_idx, int pos_gw, hipStream_t s);
hipError_t launch_ln_stats(const float* x, int N, int d, float eps, float2* stats, hipStream_t s);
hipError_t launch_ln_apply(const float* x, int N, int d, float eps, const void* g, const void* b, int w_bf16,
                           void* y, int y_f32, hipStream_t s);
hipError_t launch_rope(void* qkv, int ldqkv, int N, int heads, int hd, int is_bf16, const int4* pos3,
                       const float* inv_freq, const int* slot_axis, hipStream_t s);
// Whisper-style sinusoid position table [F, d] (fp32) and the rotary slot
// tables (inverse frequency and axis of each of the sections' slots).
hipError_t launch_sinusoid_table(float* tab, int F, int d, hipStream_t s);
hipError_t launch_rope_table(float* inv_freq, int* slot_axis, const int sections[3], float theta, hipStream_t s);
// The q | k | v biases of `layers` layers (layer l's at src + l * stride elements,
// 3 * cols / 2 values) into dst [layers, 3 cols / 2], the q and k heads
// (columns [0, cols)) in the interleaved rotary order; bf16.
hipError_t launch_rope_bias(const void* src, long stride, int layers, int cols, int hd, void* dst, hipStream_t s);
hipError_t launch_cls(const SeqMeta& m, float* x, int d, const void* cls, const void* pos0, int w_bf16,
                      hipStream_t s);
// [rows, k] 16-bit rows copied to [rows, kp] (kp % 8 == 0, dst 16-byte aligned), zero-filled past k.
hipError_t launch_pad_cols16(const void* src, int rows, int k, int kp, void* dst, hipStream_t s);
hipError_t launch_im2col_k3(const void* src, int frames_in, int C, int n_clips, int stride, int is_bf16,
                            void* dst, hipStream_t s);

struct PackArgs {
  int n;
  int cu[kMaxSeqs + 1];
  int tchw[kMaxSeqs][4];
  const float* src[kMaxSeqs];
};
hipError_t launch_pack_vision(const PackArgs& p, int cls, int merge, int patch, int tp, int K, int is_bf16,
                              void* packed, long total, hipStream_t s);
hipError_t launch_pack_audio(const PackArgs& p, int n_mels, int n_frames, int is_bf16, void* packed,
                             hipStream_t s);

}  // namespace eas

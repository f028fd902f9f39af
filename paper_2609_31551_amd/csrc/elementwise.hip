// Bandwidth-bound kernels of the Encode path: token positions, LayerNorm
// statistics / application, rotary position application, CLS insertion,
// the audio front end's im2col, and the micro-batch packers.
#include "common.h"

namespace eas {
namespace {

// (t, h, w) of token j of a t x h x w grid in storage order: merge-window
// order (2x2 windows in raster order, the window's 4 tokens consecutive) when
// merge == 2, raster order otherwise.
__device__ __forceinline__ void decode_token(int j, int h, int w, int merge, int* ti, int* hi, int* wi) {
  const int hw = h * w;
  *ti = j / hw;
  const int rem = j - *ti * hw;
  if (merge == 2) {
    const int win = rem >> 2, q = rem & 3, wb_n = w >> 1;
    *hi = 2 * (win / wb_n) + (q >> 1);
    *wi = 2 * (win % wb_n) + (q & 1);
  } else {
    *hi = rem / w;
    *wi = rem - *hi * w;
  }
}

__global__ void positions_kernel(SeqMeta m, int N, int4* pos3, int* tab_idx, int pos_gw) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  const int r = find_seq(m.cu, m.n, i);
  int j = i - m.cu[r];
  int4 p = make_int4(0, 0, 0, 0);
  if (m.cls) {
    if (j == 0) { pos3[i] = p; tab_idx[i] = 0; return; }
    j -= 1;
  }
  decode_token(j, m.thw[r][1], m.thw[r][2], m.merge, &p.x, &p.y, &p.z);
  pos3[i] = p;
  tab_idx[i] = m.cls + p.y * pos_gw + p.z;
}

__device__ __forceinline__ float wave_sum(float v) {
  // Butterfly: v += v[lane ^ o] for o = 32, 16, 8, 4, 2, 1, each lane move in
  // VALU (no LDS round trip): the two swaps pair lanes 32 and 16 apart, a
  // rotation by 8 within each 16-lane row gives lane ^ 8, shifts by 4 (the one
  // whose source stays in the row) lane ^ 4, quad permutations lane ^ 2 and
  // lane ^ 1.  Every lane ends with the same sum, summed in a fixed order.
  {
    const auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(s[0]) + __uint_as_float(s[1]);
  }
  {
    const auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(s[0]) + __uint_as_float(s[1]);
  }
  const int lane = __lane_id();
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x128, 0xF, 0xF, false));   // row_ror:8
  {
    const int up = __builtin_amdgcn_mov_dpp(__float_as_int(v), 0x104, 0xF, 0xF, false);   // row_shl:4 (lane + 4)
    const int dn = __builtin_amdgcn_mov_dpp(__float_as_int(v), 0x114, 0xF, 0xF, false);   // row_shr:4 (lane - 4)
    v += __int_as_float((lane & 4) ? dn : up);
  }
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));  // quad_perm 2,3,0,1
  v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));  // quad_perm 1,0,3,2
  return v;
}

constexpr int LN_MAXE = 32;   // elements per lane: rows up to 64 * 32 = 2048 wide

// One wave per row: mean, then the population variance of (x - mean).  The
// reduction order is fixed, so a row's statistics depend only on that row.
__device__ __forceinline__ void row_stats(const float* xr, int d, float eps, float* v, float* mu, float* rstd) {
  const int lane = threadIdx.x & 63;
  float s = 0.0f;
#pragma unroll
  for (int e = 0; e < LN_MAXE; ++e) {
    const int c = lane + 64 * e;
    v[e] = c < d ? xr[c] : 0.0f;
    s += v[e];
  }
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int e = 0; e < LN_MAXE; ++e) {
    const int c = lane + 64 * e;
    const float t = c < d ? v[e] - mean : 0.0f;
    q += t * t;
  }
  const float var = wave_sum(q) / (float)d;
  *mu = mean;
  *rstd = 1.0f / sqrtf(var + eps);
}

__global__ __launch_bounds__(256) void ln_stats_kernel(const float* x, int N, int d, float eps, float2* st) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= N) return;
  float v[LN_MAXE], mu, rstd;
  row_stats(x + (long)row * d, d, eps, v, &mu, &rstd);
  if ((threadIdx.x & 63) == 0) st[row] = make_float2(mu, rstd);
}

template <class W, class Y>
__global__ __launch_bounds__(256) void ln_apply_kernel(const float* x, int N, int d, float eps, const W* g,
                                                       const W* b, Y* y) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= N) return;
  const int lane = threadIdx.x & 63;
  float v[LN_MAXE], mu, rstd;
  row_stats(x + (long)row * d, d, eps, v, &mu, &rstd);
#pragma unroll
  for (int e = 0; e < LN_MAXE; ++e) {
    const int c = lane + 64 * e;
    if (c < d) y[(long)row * d + c] = (Y)((v[e] - mu) * rstd * (float)g[c] + (float)b[c]);
  }
}

// Vector form: one wave per row, each lane 4 consecutive elements per 16-byte
// chunk (rows with d % 4 == 0, up to 64 * 4 * LNV_MAXC wide).
constexpr int LNV_MAXC = 8;

template <class W, class Y>
__global__ __launch_bounds__(256) void ln_apply_vec_kernel(const float* x, int N, int d, float eps, const W* g,
                                                           const W* b, Y* y) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= N) return;
  const int lane = threadIdx.x & 63, nc = d >> 2;
  const float4* xr = reinterpret_cast<const float4*>(x + (long)row * d);
  // gamma and beta are fetched with the row, so their latency hides under its
  // loads and reductions (one LayerNorm over one image's 577 rows is latency-bound)
  static_assert(sizeof(W) == 2, "gamma / beta fetched as four 16-bit values per 8 bytes");
  uint2 gv[LNV_MAXC], bv[LNV_MAXC];
#pragma unroll
  for (int e = 0; e < LNV_MAXC; ++e) {
    const int c = lane + 64 * e;
    if (c < nc) {
      gv[e] = *reinterpret_cast<const uint2*>(g + 4 * c);
      bv[e] = *reinterpret_cast<const uint2*>(b + 4 * c);
    }
  }
  float4 v[LNV_MAXC];
  float s = 0.0f;
#pragma unroll
  for (int e = 0; e < LNV_MAXC; ++e) {
    const int c = lane + 64 * e;
    v[e] = c < nc ? xr[c] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    s += (v[e].x + v[e].y) + (v[e].z + v[e].w);
  }
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int e = 0; e < LNV_MAXC; ++e) {
    if (lane + 64 * e < nc) {
      const float a0 = v[e].x - mean, a1 = v[e].y - mean, a2 = v[e].z - mean, a3 = v[e].w - mean;
      q += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
    }
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + eps);
#pragma unroll
  for (int e = 0; e < LNV_MAXC; ++e) {
    const int c = lane + 64 * e;
    if (c < nc) {
      const float in[4] = {v[e].x, v[e].y, v[e].z, v[e].w};
      union { uint2 u; W h[4]; } gw, bw;
      gw.u = gv[e];
      bw.u = bv[e];
      Y out[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) out[j] = (Y)((in[j] - mean) * rstd * (float)gw.h[j] + (float)bw.h[j]);
      if constexpr (sizeof(Y) == 2) {
        union { uint2 u; Y h[4]; } o;
#pragma unroll
        for (int j = 0; j < 4; ++j) o.h[j] = out[j];
        *reinterpret_cast<uint2*>(y + (long)row * d + 4 * c) = o.u;
      } else {
        *reinterpret_cast<float4*>(y + (long)row * d + 4 * c) = make_float4(out[0], out[1], out[2], out[3]);
      }
    }
  }
}

// Rotate the pairs (k, k + hd/2) of every head of q and k in place; slot k
// turns by pos[axis(k)] * inv_freq[k].
template <class T>
__global__ void rope_kernel(T* qkv, int ldqkv, int N, int heads, int hd, const int4* pos3,
                            const float* inv_freq, const int* slot_axis) {
  const int half = hd >> 1;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const long total = (long)N * heads * half;
  if (idx >= total) return;
  const int k = (int)(idx % half);
  const int h = (int)((idx / half) % heads);
  const int i = (int)(idx / ((long)half * heads));
  const int4 p = pos3[i];
  const int ax = slot_axis[k];
  const float pos = (float)(ax == 0 ? p.x : (ax == 1 ? p.y : p.z));
  float sn, cs;
  sincosf(pos * inv_freq[k], &sn, &cs);
  const int dq = heads * hd;
#pragma unroll
  for (int part = 0; part < 2; ++part) {   // q block, then k block
    T* base = qkv + (long)i * ldqkv + part * dq + h * hd;
    const float x1 = (float)base[k], x2 = (float)base[k + half];
    base[k] = (T)(x1 * cs - x2 * sn);
    base[k + half] = (T)(x2 * cs + x1 * sn);
  }
}

// bf16 RoPE, one block per ROPE_TOK tokens: the (cos, sin) of every rotation
// slot of its tokens are computed once into LDS, then the block's threads
// rotate the (x_k, x_{k+half}) 16-byte chunk pairs of q and k, consecutive
// threads on consecutive chunks (a row's q and k heads are one contiguous
// stretch of 2 * heads * hd elements), ROPE_R pairs per thread with all their
// loads issued before the first store.  hd % 16 == 0, hd <= 128.
constexpr int ROPE_TOK = 8, ROPE_R = 5;
__global__ __launch_bounds__(256) void rope_vec_kernel(bf16* qkv, int ldqkv, int N, int heads, int hd,
                                                       const int4* pos3, const float* inv_freq, const int* slot_axis) {
  __shared__ float2 tab[ROPE_TOK * 64];   // [token][slot]: (cos, sin)
  const int half = hd >> 1, chunks = half >> 3;
  const int t0 = blockIdx.x * ROPE_TOK, nt = min(ROPE_TOK, N - t0);
  for (int e = threadIdx.x; e < nt * half; e += blockDim.x) {
    const int t = e / half, k = e % half;
    const int4 p = pos3[t0 + t];
    const int ax = slot_axis[k];
    const float pos = (float)(ax == 0 ? p.x : (ax == 1 ? p.y : p.z));
    float sn, cs;
    sincosf(pos * inv_freq[k], &sn, &cs);
    tab[t * 64 + k] = make_float2(cs, sn);
  }
  __syncthreads();
  const int per_tok = 2 * heads * chunks;   // chunk pairs of q and k per token
  const int items = nt * per_tok;
  for (int i0 = 0; i0 < items; i0 += ROPE_R * 256) {
    union { uint4 u; bf16 e[8]; } a[ROPE_R], c[ROPE_R];
    bf16* ptr[ROPE_R];
    int ti[ROPE_R], kk[ROPE_R];
#pragma unroll
    for (int r = 0; r < ROPE_R; ++r) {
      const int it = i0 + r * 256 + (int)threadIdx.x;
      ptr[r] = nullptr;
      if (it < items) {
        const int t = it / per_tok, w = it % per_tok;
        ti[r] = t;
        kk[r] = (w % chunks) * 8;
        ptr[r] = qkv + (long)(t0 + t) * ldqkv + (w / chunks) * hd + kk[r];
        a[r].u = *reinterpret_cast<const uint4*>(ptr[r]);
        c[r].u = *reinterpret_cast<const uint4*>(ptr[r] + half);
      }
    }
#pragma unroll
    for (int r = 0; r < ROPE_R; ++r) {
      if (ptr[r]) {
        const float2* f = tab + ti[r] * 64 + kk[r];
        union { uint4 u; bf16 e[8]; } oa, oc;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float2 q = f[j];
          const float x1 = (float)a[r].e[j], x2 = (float)c[r].e[j];
          oa.e[j] = (bf16)(x1 * q.x - x2 * q.y);
          oc.e[j] = (bf16)(x2 * q.x + x1 * q.y);
        }
        *reinterpret_cast<uint4*>(ptr[r]) = oa.u;
        *reinterpret_cast<uint4*>(ptr[r] + half) = oc.u;
      }
    }
  }
}

template <class W>
__global__ void cls_kernel(SeqMeta m, float* x, int d, const W* cls, const W* pos0) {
  const int r = blockIdx.x;
  for (int c = threadIdx.x; c < d; c += blockDim.x)
    x[(long)m.cu[r] * d + c] = (float)cls[c] + (float)pos0[c];
}

// dst[(clip, t), c*3 + k] = src[(clip, stride*t + k - 1), c], zero outside the
// clip: the im2col of a kernel-3, padding-1 1-D convolution over time-major
// frames, in the (channel, tap) order of a [out, C, 3] weight.
template <class T>
__global__ void im2col_k3_kernel(const T* src, int fin, int C, int fout, int stride, long total, T* dst) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int k = (int)(idx % 3);
  const int c = (int)((idx / 3) % C);
  const long row = idx / (3L * C);
  const int t = (int)(row % fout);
  const long clip = row / fout;
  const int ts = stride * t + k - 1;
  dst[idx] = (ts >= 0 && ts < fin) ? src[(clip * fin + ts) * C + c] : (T)0.0f;
}

template <class T>
__global__ void pack_vision_kernel(PackArgs p, int cls, int merge, int patch, int tp, int K, long total, T* out) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int kk = (int)(idx % K);
  const int row = (int)(idx / K);
  const int r = find_seq(p.cu, p.n, row);
  int j = row - p.cu[r];
  if (cls) {
    if (j == 0) { out[idx] = (T)0.0f; return; }
    j -= 1;
  }
  const int H = p.tchw[r][2], W = p.tchw[r][3], C = p.tchw[r][1];
  const int h = H / patch, w = W / patch;
  int ti, hi, wi;
  decode_token(j, h, w, merge, &ti, &hi, &wi);
  const int dx = kk % patch, dy = (kk / patch) % patch;
  const int tau = (kk / (patch * patch)) % tp, c = kk / (patch * patch * tp);
  const long src = (((long)(ti * tp + tau) * C + c) * H + hi * patch + dy) * W + wi * patch + dx;
  out[idx] = (T)p.src[r][src];
}

// bf16 packer: a block packs `tpb` consecutive token rows.  One thread per
// (token, c, tau, dy) line of `patch` pixels reads them as float2 pairs and
// writes the bf16 values into the block's LDS copy of the rows; the block then
// stores the rows' contiguous span with 8-byte writes, so every output line is
// written whole (patch even, every image width even, 8-byte aligned sources,
// lines <= 256, patch <= 16).
__global__ __launch_bounds__(256) void pack_vision_vec_kernel(PackArgs p, int cls, int merge, int patch, int tp, int K,
                                                              int lines, int tpb, int rows, bf16* out) {
  __shared__ __attribute__((aligned(16))) unsigned buf[256 * 16 / 2];   // tpb * K bf16
  const int row0 = blockIdx.x * tpb, nrows = min(tpb, rows - row0);
  const int t = threadIdx.x / lines, ln = threadIdx.x % lines;
  if (t < nrows) {
    const int row = row0 + t;
    unsigned* dst = buf + (t * K + ln * patch) / 2;
    const int r = find_seq(p.cu, p.n, row);
    int j = row - p.cu[r];
    if (cls && j == 0) {
      for (int x = 0; x < patch / 2; ++x) dst[x] = 0u;
    } else {
      j -= cls;
      const int dy = ln % patch, tau = (ln / patch) % tp, c = ln / (patch * tp);
      const int H = p.tchw[r][2], W = p.tchw[r][3], C = p.tchw[r][1];
      int ti, hi, wi;
      decode_token(j, H / patch, W / patch, merge, &ti, &hi, &wi);
      const float2* src = reinterpret_cast<const float2*>(
          p.src[r] + (((long)(ti * tp + tau) * C + c) * H + hi * patch + dy) * W + wi * patch);
      for (int x = 0; x < patch / 2; ++x) {
        const float2 v = src[x];
        union { unsigned u; bf16 h[2]; } o;
        o.h[0] = (bf16)v.x;
        o.h[1] = (bf16)v.y;
        dst[x] = o.u;
      }
    }
  }
  __syncthreads();
  const int n8 = nrows * K / 4;   // 8-byte pieces of the block's rows (K % 4 == 0)
  uint2* o8 = reinterpret_cast<uint2*>(out + (long)row0 * K);
  const uint2* b8 = reinterpret_cast<const uint2*>(buf);
  for (int i = threadIdx.x; i < n8; i += blockDim.x) o8[i] = b8[i];
}

// bf16 im2col for C % 8 == 0: one thread per (output frame, 8 channels) reads
// the three taps' 16-byte chunks and writes the 24 values ((channel, tap)
// order) as three 16-byte stores.
__global__ void im2col_k3_vec_kernel(const bf16* src, int fin, int C, int fout, int stride, long total, bf16* dst) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int cg = C >> 3;
  const long row = idx / cg;
  const int c0 = (int)(idx % cg) * 8;
  const int t = (int)(row % fout);
  const long clip = row / fout;
  union { uint4 u; bf16 e[8]; } in[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const int ts = stride * t + k - 1;
    in[k].u = (ts >= 0 && ts < fin) ? *reinterpret_cast<const uint4*>(src + (clip * fin + ts) * C + c0)
                                    : make_uint4(0u, 0u, 0u, 0u);
  }
  union { uint4 u[3]; bf16 e[24]; } o;
#pragma unroll
  for (int cc = 0; cc < 8; ++cc)
#pragma unroll
    for (int k = 0; k < 3; ++k) o.e[cc * 3 + k] = in[k].e[cc];
  uint4* d = reinterpret_cast<uint4*>(dst + row * 3 * C + c0 * 3);
#pragma unroll
  for (int q = 0; q < 3; ++q) d[q] = o.u[q];
}

// [n_mels, n_frames] -> [n_frames, n_mels] per clip.
template <class T>
__global__ void pack_audio_kernel(PackArgs p, int n_mels, int n_frames, T* out) {
  const long per = (long)n_mels * n_frames;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= per * p.n) return;
  const int clip = (int)(idx / per);
  const long e = idx % per;
  const int t = (int)(e / n_mels), mel = (int)(e % n_mels);
  out[idx] = (T)p.src[clip][(long)mel * n_frames + t];
}

// [rows, k] 16-bit elements -> [rows, kp] with zero columns k .. kp; a thread
// writes one 16-byte chunk of the output.
__global__ void pad_cols16_kernel(const uint16_t* src, int rows, int k, int kp, uint16_t* dst) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const int cpr = kp / 8;
  if (idx >= (long)rows * cpr) return;
  const int r = (int)(idx / cpr), c0 = (int)(idx % cpr) * 8;
  union { uint4 u; uint16_t h[8]; } o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o.h[e] = c0 + e < k ? src[(long)r * k + c0 + e] : (uint16_t)0;
  *reinterpret_cast<uint4*>(dst + (long)r * kp + c0) = o.u;
}

inline unsigned blocks_for(long n, int bs) { return (unsigned)((n + bs - 1) / bs); }

}  // namespace

namespace {

// Whisper-style sinusoid table [F, d]: columns i < d/2 hold sin(t * w_i) and
// columns d/2 + i hold cos(t * w_i), w_i = exp(-i ln(10^4) / (d/2 - 1));
// evaluated in double, stored as fp32.
__global__ void sinusoid_table_kernel(float* tab, int F, int d) {
  const int hc = d / 2;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)F * hc) return;
  const int t = (int)(idx / hc), i = (int)(idx % hc);
  const double a = (double)t * exp(-log(10000.0) / (double)(hc - 1) * (double)i);
  tab[(long)t * d + i] = (float)sin(a);
  tab[(long)t * d + hc + i] = (float)cos(a);
}

// Rotary slot tables: the sections s0, s1, s2 of slots turn with the t, h
// and w position; slot j of an axis with n slots turns by theta^(-j / n).
__global__ void rope_table_kernel(float* inv_freq, int* slot_axis, int s0, int s1, int s2, float theta) {
  const int k = threadIdx.x;
  if (k >= s0 + s1 + s2) return;
  const int ax = k < s0 ? 0 : (k < s0 + s1 ? 1 : 2);
  const int j = k - (ax == 0 ? 0 : (ax == 1 ? s0 : s0 + s1));
  const int n = ax == 0 ? s0 : (ax == 1 ? s1 : s2);
  inv_freq[k] = (float)pow((double)theta, -(double)j / (double)n);
  slot_axis[k] = ax;
}

// dst[l, n] = src[l * stride + rope_src_row(n)]: every layer's q | k | v bias with
// the q and k heads interleaved for the rotary epilogue.
__global__ void rope_bias_kernel(const bf16* src, long stride, int w, int cols, int hd, unsigned hd_inv, bf16* dst,
                                 long total) {
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int l = (int)(idx / w), n = (int)(idx % w);
  dst[idx] = src[l * stride + rope_src_row(n, hd, hd_inv, cols)];
}

}  // namespace

hipError_t launch_rope_bias(const void* src, long stride, int layers, int cols, int hd, void* dst, hipStream_t s) {
  const int w = cols / 2 * 3;
  const long total = (long)layers * w;
  if (cols % 2 || hd % 2 || hd > 128 || cols % hd || w >= 65536) return hipErrorInvalidValue;
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_bias_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, s, static_cast<const bf16*>(src),
                     stride, w, cols, hd, rope_hd_inv(hd), static_cast<bf16*>(dst), total);
  return hipGetLastError();
}

hipError_t launch_sinusoid_table(float* tab, int F, int d, hipStream_t s) {
  if (d < 4 || d % 2) return hipErrorInvalidValue;
  const long total = (long)F * (d / 2);
  if (total == 0) return hipSuccess;
  hipLaunchKernelGGL(sinusoid_table_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, s, tab, F, d);
  return hipGetLastError();
}

hipError_t launch_rope_table(float* inv_freq, int* slot_axis, const int sections[3], float theta, hipStream_t s) {
  if (sections[0] + sections[1] + sections[2] > 256) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rope_table_kernel, dim3(1), dim3(256), 0, s, inv_freq, slot_axis, sections[0], sections[1],
                     sections[2], theta);
  return hipGetLastError();
}

hipError_t launch_positions(const SeqMeta& m, int N, int4* pos3, int* tab_idx, int pos_gw, hipStream_t s) {
  hipLaunchKernelGGL(positions_kernel, dim3(blocks_for(N, 256)), dim3(256), 0, s, m, N, pos3, tab_idx, pos_gw);
  return hipGetLastError();
}

hipError_t launch_ln_stats(const float* x, int N, int d, float eps, float2* stats, hipStream_t s) {
  if (d > 64 * LN_MAXE) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ln_stats_kernel, dim3(blocks_for(N, 4)), dim3(256), 0, s, x, N, d, eps, stats);
  return hipGetLastError();
}

hipError_t launch_ln_apply(const float* x, int N, int d, float eps, const void* g, const void* b, int w_bf16,
                           void* y, int y_f32, hipStream_t s) {
  if (d > 64 * LN_MAXE) return hipErrorInvalidValue;
  const dim3 grid(blocks_for(N, 4)), blk(256);
  const bool al = (uintptr_t)x % 16 == 0 && (uintptr_t)y % (y_f32 ? 16 : 8) == 0 &&
                  (uintptr_t)g % (w_bf16 ? 8 : 16) == 0 && (uintptr_t)b % (w_bf16 ? 8 : 16) == 0;
  if (d % 4 == 0 && d <= 256 * LNV_MAXC && al && w_bf16) {
    if (y_f32)
      hipLaunchKernelGGL((ln_apply_vec_kernel<bf16, float>), grid, blk, 0, s, x, N, d, eps, (const bf16*)g,
                         (const bf16*)b, (float*)y);
    else
      hipLaunchKernelGGL((ln_apply_vec_kernel<bf16, bf16>), grid, blk, 0, s, x, N, d, eps, (const bf16*)g,
                         (const bf16*)b, (bf16*)y);
    return hipGetLastError();
  }
  if (w_bf16 && y_f32)
    hipLaunchKernelGGL((ln_apply_kernel<bf16, float>), grid, blk, 0, s, x, N, d, eps, (const bf16*)g, (const bf16*)b, (float*)y);
  else if (w_bf16)
    hipLaunchKernelGGL((ln_apply_kernel<bf16, bf16>), grid, blk, 0, s, x, N, d, eps, (const bf16*)g, (const bf16*)b, (bf16*)y);
  else if (y_f32)
    hipLaunchKernelGGL((ln_apply_kernel<float, float>), grid, blk, 0, s, x, N, d, eps, (const float*)g, (const float*)b, (float*)y);
  else
    hipLaunchKernelGGL((ln_apply_kernel<float, bf16>), grid, blk, 0, s, x, N, d, eps, (const float*)g, (const float*)b, (bf16*)y);
  return hipGetLastError();
}

hipError_t launch_rope(void* qkv, int ldqkv, int N, int heads, int hd, int is_bf16, const int4* pos3,
                       const float* inv_freq, const int* slot_axis, hipStream_t s) {
  const long total = (long)N * heads * (hd / 2);
  if (is_bf16 && hd % 16 == 0 && hd <= 128 && ldqkv % 8 == 0 && (uintptr_t)qkv % 16 == 0) {
    if (N == 0) return hipSuccess;
    hipLaunchKernelGGL(rope_vec_kernel, dim3((N + ROPE_TOK - 1) / ROPE_TOK), dim3(256), 0, s, (bf16*)qkv, ldqkv, N,
                       heads, hd, pos3, inv_freq, slot_axis);
    return hipGetLastError();
  }
  if (is_bf16)
    hipLaunchKernelGGL((rope_kernel<bf16>), dim3(blocks_for(total, 256)), dim3(256), 0, s, (bf16*)qkv, ldqkv, N,
                       heads, hd, pos3, inv_freq, slot_axis);
  else
    hipLaunchKernelGGL((rope_kernel<float>), dim3(blocks_for(total, 256)), dim3(256), 0, s, (float*)qkv, ldqkv, N,
                       heads, hd, pos3, inv_freq, slot_axis);
  return hipGetLastError();
}

hipError_t launch_pad_cols16(const void* src, int rows, int k, int kp, void* dst, hipStream_t s) {
  if (kp % 8 || kp < k || (uintptr_t)dst % 16) return hipErrorInvalidValue;
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(pad_cols16_kernel, dim3(blocks_for((long)rows * (kp / 8), 256)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(src), rows, k, kp, static_cast<uint16_t*>(dst));
  return hipGetLastError();
}

hipError_t launch_cls(const SeqMeta& m, float* x, int d, const void* cls, const void* pos0, int w_bf16, hipStream_t s) {
  if (w_bf16)
    hipLaunchKernelGGL((cls_kernel<bf16>), dim3(m.n), dim3(256), 0, s, m, x, d, (const bf16*)cls, (const bf16*)pos0);
  else
    hipLaunchKernelGGL((cls_kernel<float>), dim3(m.n), dim3(256), 0, s, m, x, d, (const float*)cls, (const float*)pos0);
  return hipGetLastError();
}

hipError_t launch_im2col_k3(const void* src, int frames_in, int C, int n_clips, int stride, int is_bf16, void* dst,
                            hipStream_t s) {
  const int fout = (frames_in - 1) / stride + 1;
  const long total = (long)n_clips * fout * C * 3;
  if (total == 0) return hipSuccess;
  if (is_bf16 && C % 8 == 0 && (uintptr_t)src % 16 == 0 && (uintptr_t)dst % 16 == 0) {
    const long threads = (long)n_clips * fout * (C / 8);
    hipLaunchKernelGGL(im2col_k3_vec_kernel, dim3(blocks_for(threads, 256)), dim3(256), 0, s, (const bf16*)src,
                       frames_in, C, fout, stride, threads, (bf16*)dst);
    return hipGetLastError();
  }
  if (is_bf16)
    hipLaunchKernelGGL((im2col_k3_kernel<bf16>), dim3(blocks_for(total, 256)), dim3(256), 0, s, (const bf16*)src,
                       frames_in, C, fout, stride, total, (bf16*)dst);
  else
    hipLaunchKernelGGL((im2col_k3_kernel<float>), dim3(blocks_for(total, 256)), dim3(256), 0, s, (const float*)src,
                       frames_in, C, fout, stride, total, (float*)dst);
  return hipGetLastError();
}

hipError_t launch_pack_vision(const PackArgs& p, int cls, int merge, int patch, int tp, int K, int is_bf16,
                              void* packed, long total, hipStream_t s) {
  if (total == 0) return hipSuccess;
  const int lines = K / patch;
  bool vec = is_bf16 && patch % 2 == 0 && patch <= 16 && lines <= 256 && (uintptr_t)packed % 8 == 0;
  for (int r = 0; vec && r < p.n; ++r) vec = p.tchw[r][3] % 2 == 0 && (uintptr_t)p.src[r] % 8 == 0;
  if (vec) {
    const int rows = (int)(total / K), tpb = 256 / lines;
    hipLaunchKernelGGL(pack_vision_vec_kernel, dim3((rows + tpb - 1) / tpb), dim3(256), 0, s, p, cls, merge, patch, tp,
                       K, lines, tpb, rows, (bf16*)packed);
    return hipGetLastError();
  }
  if (is_bf16)
    hipLaunchKernelGGL((pack_vision_kernel<bf16>), dim3(blocks_for(total, 256)), dim3(256), 0, s, p, cls, merge, patch,
                       tp, K, total, (bf16*)packed);
  else
    hipLaunchKernelGGL((pack_vision_kernel<float>), dim3(blocks_for(total, 256)), dim3(256), 0, s, p, cls, merge,
                       patch, tp, K, total, (float*)packed);
  return hipGetLastError();
}

hipError_t launch_pack_audio(const PackArgs& p, int n_mels, int n_frames, int is_bf16, void* packed, hipStream_t s) {
  const long total = (long)p.n * n_mels * n_frames;
  if (is_bf16)
    hipLaunchKernelGGL((pack_audio_kernel<bf16>), dim3(blocks_for(total, 256)), dim3(256), 0, s, p, n_mels, n_frames,
                       (bf16*)packed);
  else
    hipLaunchKernelGGL((pack_audio_kernel<float>), dim3(blocks_for(total, 256)), dim3(256), 0, s, p, n_mels, n_frames,
                       (float*)packed);
  return hipGetLastError();
}

}  // namespace eas

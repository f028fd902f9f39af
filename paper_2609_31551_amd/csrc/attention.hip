// Variable-length block-diagonal attention over packed sequences:
// for every sequence r (tokens cu[r] .. cu[r+1]) and head h,
//   O = softmax(Q K^T / sqrt(hd)) V,
// full (non-causal) within the sequence, nothing across sequences.
//
// bf16 MFMA kernel (gfx950).  A workgroup of 4 waves owns 128 queries of one
// (sequence, head); each wave owns 32 of them.  Keys stream through LDS in
// tiles of 64 anchored at the sequence start, so a query's result does not
// depend on where its sequence sits in the micro-batch.  Per key tile:
//  * S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (K rows from LDS as the A
//    operand, the wave's Q held in registers as the B operand).  In the S^T
//    accumulator lane l holds 16 scores of query l % 32, so the online
//    softmax (running max, rescale, exp2) is lane-local apart from one
//    cross-half shuffle for the max (lanes l and l ^ 32 share a query).
//  * O^T += V^T P^T: the bf16-rounded probabilities already sit in the
//    B-operand layout, and V is stored transposed in LDS so each lane reads
//    its V^T operand with two 8-byte loads.  O^T keeps lane l on query l % 32,
//    so the softmax rescale of O is lane-local too.
// Softmax runs in fp32 on exp2 with the 1/sqrt(hd) * log2(e) scale folded in.
#include "common.h"

namespace eas {
namespace {

constexpr int QT = 128;   // queries per workgroup (bf16 kernel)
constexpr int KT = 64;    // keys per LDS tile

__device__ __forceinline__ void decode_tile(const AttnWork& w, int tile, int qt_size, int* s0, int* s1, int* q0) {
  int i = 0;
  while (i + 1 < w.n && w.tile_start[i + 1] <= tile) ++i;
  const int r = w.order[i];
  *s0 = w.cu[r];
  *s1 = w.cu[r + 1];
  *q0 = *s0 + (tile - w.tile_start[i]) * qt_size;
}

template <int HD>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnArgs a, AttnWork w) {
  constexpr int KS = HD / 16;          // 16-wide k-steps of Q K^T
  constexpr int HB = (HD + 31) / 32;   // 32-row blocks of O^T
  constexpr int LDKS = HD + 8;         // K tile row stride (bf16)
  constexpr int LDV = KT + 4;          // V^T tile row stride (bf16), 8-byte aligned rows
  __shared__ __attribute__((aligned(16))) bf16 Ks[KT * LDKS];
  __shared__ __attribute__((aligned(16))) bf16 Vt[HB * 32 * LDV];

  const int h = blockIdx.x % a.heads;
  int s0, s1, q0;
  decode_tile(w, blockIdx.x / a.heads, QT, &s0, &s1, &q0);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 5, l32 = lane & 31;
  const int dq = a.heads * HD;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const float c = a.scale * 1.4426950408889634f;

  // this wave's 32 queries (rows past the sequence end are clamped, never stored)
  const int qi = q0 + wave * 32 + l32;
  const int qr = qi < s1 ? qi : s1 - 1;
  bf16x8 qf[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks)
    qf[ks] = *reinterpret_cast<const bf16x8*>(qkv + (long)qr * a.ldqkv + h * HD + ks * 16 + g * 8);

  f32x16 o[HB];
#pragma unroll
  for (int hb = 0; hb < HB; ++hb)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[hb][e] = 0.0f;
  float m_run = -INFINITY, l_part = 0.0f;

  for (int k0 = s0; k0 < s1; k0 += KT) {
    __syncthreads();
    // K tile [64 keys][HD], zero past the sequence end
    for (int cidx = tid; cidx < KT * (HD / 8); cidx += 256) {
      const int key = cidx / (HD / 8), dc = (cidx % (HD / 8)) * 8;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (k0 + key < s1) v = *reinterpret_cast<const uint4*>(qkv + (long)(k0 + key) * a.ldqkv + dq + h * HD + dc);
      *reinterpret_cast<uint4*>(Ks + key * LDKS + dc) = v;
    }
    // V tile, transposed: Vt[d][key]; each thread moves two keys x 8 dims
    for (int cidx = tid; cidx < (KT / 2) * (HD / 8); cidx += 256) {
      const int kp = cidx % (KT / 2), dc = (cidx / (KT / 2)) * 8;
      union { uint4 u; bf16 h[8]; } v0, v1;
      v0.u = make_uint4(0, 0, 0, 0);
      v1.u = make_uint4(0, 0, 0, 0);
      const int key = k0 + 2 * kp;
      if (key < s1) v0.u = *reinterpret_cast<const uint4*>(qkv + (long)key * a.ldqkv + 2 * dq + h * HD + dc);
      if (key + 1 < s1) v1.u = *reinterpret_cast<const uint4*>(qkv + (long)(key + 1) * a.ldqkv + 2 * dq + h * HD + dc);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        union { uint32_t u; bf16 h[2]; } pr;
        pr.h[0] = v0.h[e];
        pr.h[1] = v1.h[e];
        *reinterpret_cast<uint32_t*>(Vt + (dc + e) * LDV + 2 * kp) = pr.u;
      }
    }
    __syncthreads();

    // S^T blocks: keys kb*32 .. +32 of this tile x the wave's 32 queries
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int e = 0; e < 16; ++e) s[kb][e] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(Ks + (kb * 32 + l32) * LDKS + ks * 16 + g * 8);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[kb], 0, 0, 0);
      }
    }
    // scale, mask, running max
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = k0 + kb * 32 + (e >> 2) * 8 + g * 4 + (e & 3);
        const float v = key < s1 ? s[kb][e] * c : -INFINITY;
        s[kb][e] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.0f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const float p = exp2f(s[kb][e] - m_new);
        s[kb][e] = p;
        psum += p;
      }
    l_part = l_part * alpha + psum;
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[hb][e] *= alpha;

    // O^T += V^T P^T over 4 chunks of 16 keys
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int ch = 0; ch < 2; ++ch) {
        bf16x8 pb;
#pragma unroll
        for (int i = 0; i < 8; ++i) pb[i] = (bf16)s[kb][8 * ch + i];
        const int kofs = kb * 32 + 16 * ch + 4 * g;
#pragma unroll
        for (int hb = 0; hb < HB; ++hb) {
          int d = hb * 32 + l32;
          d = d < HD ? d : 0;   // padding rows of the last block read a real row; their output is dropped
          const bf16* vp = Vt + d * LDV + kofs;
          union { bf16x8 v; uint2 u[2]; } va;
          va.u[0] = *reinterpret_cast<const uint2*>(vp);
          va.u[1] = *reinterpret_cast<const uint2*>(vp + 8);
          o[hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va.v, pb, o[hb], 0, 0, 0);
        }
      }
  }

  const float l_tot = l_part + __shfl_xor(l_part, 32, 64);
  const float inv = 1.0f / l_tot;
  if (qi < s1) {
    bf16* out = static_cast<bf16*>(a.out) + (long)qi * a.ldo + h * HD;
#pragma unroll
    for (int hb = 0; hb < HB; ++hb)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int d = hb * 32 + e4 * 8 + g * 4;
        if (d < HD) {
          union { uint2 u; bf16 h[4]; } st;
#pragma unroll
          for (int e = 0; e < 4; ++e) st.h[e] = (bf16)(o[hb][e4 * 4 + e] * inv);
          *reinterpret_cast<uint2*>(out + d) = st.u;
        }
      }
  }
}

// fp32 kernel: one thread per query, 64 queries per workgroup, key/value tiles
// of 64 through LDS, online softmax key by key.
constexpr int QT32 = 64;

template <int HD>
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a, AttnWork w) {
  __shared__ float Ks[KT][HD + 1];
  __shared__ float Vs[KT][HD + 1];
  const int h = blockIdx.x % a.heads;
  int s0, s1, q0;
  decode_tile(w, blockIdx.x / a.heads, QT32, &s0, &s1, &q0);
  const int tid = threadIdx.x;
  const int dq = a.heads * HD;
  const float* qkv = static_cast<const float*>(a.qkv);
  const int qi = q0 + tid;
  const int qr = qi < s1 ? qi : s1 - 1;
  float q[HD], o[HD];
#pragma unroll
  for (int d = 0; d < HD; ++d) {
    q[d] = qkv[(long)qr * a.ldqkv + h * HD + d] * a.scale;
    o[d] = 0.0f;
  }
  float m = -INFINITY, l = 0.0f;
  for (int k0 = s0; k0 < s1; k0 += KT) {
    __syncthreads();
    for (int e = tid; e < KT * HD; e += 64) {
      const int key = e / HD, d = e % HD;
      const bool in = k0 + key < s1;
      Ks[key][d] = in ? qkv[(long)(k0 + key) * a.ldqkv + dq + h * HD + d] : 0.0f;
      Vs[key][d] = in ? qkv[(long)(k0 + key) * a.ldqkv + 2 * dq + h * HD + d] : 0.0f;
    }
    __syncthreads();
    const int nk = min(KT, s1 - k0);
    for (int j = 0; j < nk; ++j) {
      float sc = 0.0f;
#pragma unroll
      for (int d = 0; d < HD; ++d) sc = fmaf(q[d], Ks[j][d], sc);
      const float m_new = fmaxf(m, sc);
      const float alpha = expf(m - m_new), p = expf(sc - m_new);
      l = l * alpha + p;
#pragma unroll
      for (int d = 0; d < HD; ++d) o[d] = fmaf(p, Vs[j][d], o[d] * alpha);
      m = m_new;
    }
  }
  if (qi < s1) {
    float* out = static_cast<float*>(a.out) + (long)qi * a.ldo + h * HD;
#pragma unroll
    for (int d = 0; d < HD; ++d) out[d] = o[d] / l;
  }
}

}  // namespace

int attention_q_tile(int dtype_bf16) { return dtype_bf16 ? QT : QT32; }

hipError_t launch_attention_bf16(const AttnArgs& a, const AttnWork& w, int total_tiles, int N, hipStream_t s,
                                 const char** kname) {
  // head_dim 64 and 80 always take the DMA kernel: the library caps a handle's
  // tokens so that its 32-bit offsets hold, and keeps the qkv rows 16-byte
  // aligned, so one kernel (one summation order) serves every micro-batch
  if (a.hd == 64 || a.hd == 80)
    return attention_dma_supported(a, N) ? launch_attention_bf16_dma(a, w, total_tiles, s, kname)
                                         : hipErrorInvalidValue;
  const dim3 grid((unsigned)(total_tiles * a.heads)), blk(256);
  switch (a.hd) {
    case 128: *kname = "attn_bf16_hd128"; hipLaunchKernelGGL((attn_bf16_kernel<128>), grid, blk, 0, s, a, w); break;
    case 16: *kname = "attn_bf16_hd16"; hipLaunchKernelGGL((attn_bf16_kernel<16>), grid, blk, 0, s, a, w); break;
    case 32: *kname = "attn_bf16_hd32"; hipLaunchKernelGGL((attn_bf16_kernel<32>), grid, blk, 0, s, a, w); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_attention_f32(const AttnArgs& a, const AttnWork& w, int total_tiles, hipStream_t s,
                                const char** kname) {
  const dim3 grid((unsigned)(total_tiles * a.heads)), blk(64);
  switch (a.hd) {
    case 16: *kname = "attn_f32_hd16"; hipLaunchKernelGGL((attn_f32_kernel<16>), grid, blk, 0, s, a, w); break;
    case 32: *kname = "attn_f32_hd32"; hipLaunchKernelGGL((attn_f32_kernel<32>), grid, blk, 0, s, a, w); break;
    case 64: *kname = "attn_f32_hd64"; hipLaunchKernelGGL((attn_f32_kernel<64>), grid, blk, 0, s, a, w); break;
    case 80: *kname = "attn_f32_hd80"; hipLaunchKernelGGL((attn_f32_kernel<80>), grid, blk, 0, s, a, w); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace eas

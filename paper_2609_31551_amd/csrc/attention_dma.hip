// Variable-length block-diagonal attention, bf16 MFMA, head_dim 64 or 80 --
// the form that carries the CLIP, Qwen-ViT and Whisper encoders.
//
// For every sequence r (tokens cu[r] .. cu[r+1]) and head h:
//   O = softmax(Q K^T / sqrt(hd)) V, full within the sequence, nothing across.
//
// Design (gfx950):
//  * A workgroup is 4 or 8 waves and owns 128 or 256 queries of one
//    (sequence, head); each wave owns one 32-query MFMA column block (<= 128
//    VGPRs, so 4 waves share a SIMD and hide each other's latency).  The
//    256-query form shares every K / V tile among twice the queries, which
//    halves the DMA traffic per score; it is taken for head_dim 80 when the
//    coarser tiles add almost no query slots.
//  * K and V tiles of 64 keys arrive by direct DMA (global_load_lds_dwordx4)
//    into two LDS buffers: tile t+1 streams in while tile t is consumed,
//    one barrier per tile.  Tiles are anchored at the sequence start; rows
//    past its end re-read the last row and are masked out of the softmax.
//  * Both tiles are stored row-major with a per-row rotation of the 16-byte
//    chunks (2(r&3) + ((r>>2)&1) for 8-chunk rows, (r>>2)&1 for 10-chunk
//    rows), which keeps the transposing V reads free of bank conflicts; the
//    K reads see at most 2-way conflicts (a conflict-free K order measured
//    no faster).
//  * S^T = K Q^T (K rows as the A operand, Q in registers as the B operand):
//    lane l holds 16 scores of query l % 32, so the online softmax is
//    lane-local except one cross-half shuffle for the running max.
//  * O^T += V^T P^T: the bf16-rounded probabilities already sit in the B
//    operand layout; the V^T operand comes straight from the row-major V
//    tile through ds_read_b64_tr_b16, whose 16-lane transpose turns four
//    8-byte row pieces into four columns.
//  * For head_dim 64, both halves' S^T MFMAs of a 64-key tile are issued
//    before the first softmax, so the softmax of one half overlaps MFMAs of
//    the other; head_dim 80 keeps one half's scores live at a time.
//  * A 32-key half tile that lies wholly past the sequence end is skipped,
//    and a wave whose queries all lie past the end skips the arithmetic.
#include "common.h"

namespace eas {
namespace {

// keys per K / V tile
constexpr int KTILE = 64;

#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(unsigned lds_addr, unsigned voff, const void* gbase) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2\n"
               :: "s"(lds_addr), "v"(voff), "s"(gbase) : "memory", "m0");
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

template <int HD, int QB_, int QT_>
struct AttnCfg {
  static constexpr int QT = QT_;                   // queries per workgroup
  static constexpr int QB = QB_;                   // 32-query blocks per wave
  static constexpr int NW = QT / (32 * QB);        // waves per workgroup
  static constexpr int R = HD / 8;                 // 16-byte chunks per K / V row
  static constexpr int KS = HD / 16;               // 16-wide k-steps of Q K^T
  static constexpr int HB = (HD + 31) / 32;        // 32-row blocks of O^T
  static constexpr int TILE = KTILE * R * 16;      // bytes of one K or V tile
  static constexpr int BUF = 2 * TILE;             // K + V
  static constexpr int NDMA = TILE / 1024;         // DMA instructions per operand per tile (= R)
  static constexpr int DMA = (NDMA + NW - 1) / NW; // per wave (instruction wave + NW*j)
  // Register budget for 4 waves per SIMD (<= 128 VGPRs): head_dim 64 issues both
  // halves' S^T MFMAs ahead of the softmax (a second score block per query
  // block); head_dim 80 instead reads each 16-key chunk's V^T fragments right
  // before its MFMAs.
  static constexpr bool OVERLAP = HD <= 64;
  static constexpr bool V_DIRECT = HD > 64;
  // The last O^T block has HB*32 - HD padding rows (16 for head_dim 80): fed
  // with ones instead of V, they accumulate each query's softmax row sum in
  // the MFMA (element 8 of every lane lands on row HD or HD + 4).
  static constexpr bool MFMA_SUM = HB * 32 - HD >= 16;
  __device__ static int rot(int row) { return R == 8 ? 2 * (row & 3) + ((row >> 2) & 1) : ((row >> 2) & 1); }
  // logical chunk L of row `row` sits at physical chunk phys(row, L)
  __device__ static int phys(int row, int L) { return (L + rot(row)) % R; }
  __device__ static int logical(int row, int p) { return (p + R - rot(row)) % R; }
};

__device__ __forceinline__ void decode(const AttnWork& w, int tile, int qt, int* s0, int* s1, int* q0) {
  int i = 0;
  while (i + 1 < w.n && w.tile_start[i + 1] <= tile) ++i;
  const int r = w.order[i];
  *s0 = w.cu[r];
  *s1 = w.cu[r + 1];
  *q0 = *s0 + (tile - w.tile_start[i]) * qt;
}

// Held to 128 VGPRs (4 waves per SIMD) explicitly: left to itself the register
// allocator takes 130 (head_dim 80, and 64 with the staged output) and loses a
// wave per SIMD
template <int HD, int QB, int QT>
__global__ __launch_bounds__(QT / QB * 2)
__attribute__((amdgpu_waves_per_eu(4, HD > 64 ? 4 : 8)))
void attn_bf16_dma_kernel(AttnArgs a, AttnWork w) {
  using C = AttnCfg<HD, QB, QT>;
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const unsigned lds0 = (unsigned)(size_t)((__attribute__((address_space(3))) char*)smem);
  const int h = blockIdx.x % a.heads;
  int s0, s1, q0;
  decode(w, blockIdx.x / a.heads, C::QT, &s0, &s1, &q0);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 5, l32 = lane & 31;
  const int dq = a.heads * HD;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const float c = a.scale * 1.4426950408889634f;
  const int qw0 = q0 + wave * 32 * QB;       // this wave's first query
  const bool active = qw0 < s1;              // uniform per wave

  // ---- DMA of one K + V tile: DMA instruction q (1 KB = 64 slots) belongs to
  // wave q % NW; slot s of a tile is 16 bytes at s*16: row s / R, physical
  // chunk s % R.
  int drow[C::DMA], dcol[C::DMA];
#pragma unroll
  for (int j = 0; j < C::DMA; ++j) {
    const int slot = min(wave + C::NW * j, C::NDMA - 1) * 64 + lane;
    drow[j] = slot / C::R;
    dcol[j] = h * HD + C::logical(drow[j], slot % C::R) * 8;
  }
  auto issue = [&](int k0, int buf) {
    const unsigned base = lds0 + buf * C::BUF;
#pragma unroll
    for (int j = 0; j < C::DMA; ++j) {
      const int q = wave + C::NW * j;
      if (C::NDMA % C::NW == 0 || q < C::NDMA) {
        const long key = min(k0 + drow[j], s1 - 1);
        dma16(base + q * 1024, (unsigned)((key * a.ldqkv + dq + dcol[j]) * 2), qkv);
        dma16(base + C::TILE + q * 1024, (unsigned)((key * a.ldqkv + 2 * dq + dcol[j]) * 2), qkv);
      }
    }
  };

  // Q fragments: query block qb, k-step ks: lane l holds hd ks*16 + g*8 .. +8 of query l%32
  bf16x8 qf[QB][C::KS];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qr = min(qw0 + qb * 32 + l32, s1 - 1);
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks)
      qf[qb][ks] = *reinterpret_cast<const bf16x8*>(qkv + (long)qr * a.ldqkv + h * HD + ks * 16 + g * 8);
  }
  // consume the Q loads here, before any DMA is in flight, so the compiler's
  // own wait for them cannot also wait on a prefetch
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) asm volatile("" :: "v"(qf[qb][ks]));

  f32x16 o[QB][C::HB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int hb = 0; hb < C::HB; ++hb)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[qb][hb][e] = 0.0f;
  float m_run[QB], l_part[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) { m_run[qb] = 0.0f; l_part[qb] = 0.0f; }

  // K operand reads: row kb*32 + l32, logical chunk 2ks + g (the rotation only
  // depends on row & 7, i.e. on l32)
  int kofs[C::KS];
#pragma unroll
  for (int ks = 0; ks < C::KS; ++ks) kofs[ks] = l32 * C::R * 16 + C::phys(l32, 2 * ks + g) * 16;
  // V^T operand reads: lane 16q + 4e + t reads row 32kb + 16ch + 8half + 4g + e,
  // columns hb*32 + 16(q%2) + 4t .. +4; the row's rotation depends only on (g, e)
  const int vq = lane >> 4, ve = (lane >> 2) & 3, vt = lane & 3;
  const int vrow = 4 * g + ve;
  int vofs[C::HB];
#pragma unroll
  for (int hb = 0; hb < C::HB; ++hb) {
    int col = hb * 32 + 16 * (vq & 1) + 4 * vt;
    if (col >= HD) col -= 16;   // padding rows of the last O^T block: any real column, result dropped
    vofs[hb] = vrow * C::R * 16 + C::phys(vrow, col >> 3) * 16 + (col & 7) * 2;
  }
  __attribute__((address_space(3))) char* lds = (__attribute__((address_space(3))) char*)smem;

  const int ntiles = (s1 - s0 + KTILE - 1) / KTILE;
  issue(s0, 0);
  for (int t = 0; t < ntiles; ++t) {
    const int k0 = s0 + t * KTILE, buf = t & 1;
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");   // tile t landed; reads of t-1 done
    __syncthreads();
    if (t + 1 < ntiles) issue(k0 + KTILE, buf ^ 1);
    if (!active) continue;
    const char* Kt = smem + buf * C::BUF;
    const int nkb = k0 + 32 < s1 ? 2 : 1;   // 32-key halves holding at least one key

    // Per 32-key half kb: S^T = K Q^T, online softmax, O^T += V^T P^T.  Both
    // halves' S^T MFMAs are issued first, so the first half's softmax (VALU)
    // runs while the second half's MFMAs execute, and the second half's
    // softmax overlaps the first half's P V MFMAs.
    auto scores = [&](int kb, f32x16* sc) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[qb][e] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(Kt + kb * 32 * C::R * 16 + kofs[ks]);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          sc[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[qb][ks], sc[qb], 0, 0, 0);
      }
    };
    // lanes whose V^T fragment rows lie past HD in the last block (MFMA_SUM)
    const bool pad_lane = C::MFMA_SUM && (lane & 31) >= HD - (C::HB - 1) * 32;
    bf16x8 ones;
#pragma unroll
    for (int e = 0; e < 8; ++e) ones[e] = (bf16)1.0f;
    // V^T operand fragments of half kb: [ch][hb], 16 keys each
    auto read_v = [&](int kb, bf16x8 (*va)[C::HB]) {
#pragma unroll
      for (int ch = 0; ch < 2; ++ch)
#pragma unroll
        for (int hb = 0; hb < C::HB; ++hb) {
          union { bf16x8 v; v4i16 h[2]; } u;
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const int rbase = (kb * 32 + 16 * ch + 8 * half) * C::R * 16;
            u.h[half] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_v4i16*)(lds + buf * C::BUF + C::TILE + rbase + vofs[hb]));
          }
          va[ch][hb] = (hb == C::HB - 1 && pad_lane) ? ones : u.v;
        }
    };
    // Online softmax.  Scores are masked only in a half that reaches past the
    // sequence end.  One FMA turns each score into x = s*c - m, log2 units
    // relative to the running max m (scale folded in), and the max is taken
    // over x.  m is raised lazily: O and the row sum keep a stale m until some
    // x exceeds 8, so p = 2^x <= 256 and the rescale of O is usually skipped;
    // both share m, so O / sum is unchanged.  m starts at 0, and the first
    // half tile (`first`) always sets it to that tile's max.
    auto softmax = [&](int kb, bool first, f32x16* sc, bf16x8 (*pb)[2]) {
      const int kh = k0 + kb * 32;
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const float nm = -m_run[qb];
#pragma unroll
        for (int e = 0; e < 16; ++e) sc[qb][e] = fmaf(sc[qb][e], c, nm);
      }
      if (kh + 32 > s1) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (kh + (e >> 2) * 8 + g * 4 + (e & 3) >= s1) sc[qb][e] = -INFINITY;
      }
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        float mx = sc[qb][0];
#pragma unroll
        for (int e = 1; e < 16; ++e) mx = fmaxf(mx, sc[qb][e]);
        {   // both 16-key halves of query l % 32: lanes l and l ^ 32, swapped in VALU
          const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
          mx = fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
        }
        const bool need = first || mx > 8.0f;
        if (__any(need)) {
          const float d = need ? mx : 0.0f;   // m rises by d
          const float alpha = first ? 0.0f : __builtin_amdgcn_exp2f(-d);   // O and l are still 0 at first
          m_run[qb] += d;
          l_part[qb] *= alpha;
#pragma unroll
          for (int hb = 0; hb < C::HB; ++hb)
#pragma unroll
            for (int e = 0; e < 16; ++e) o[qb][hb][e] *= alpha;
#pragma unroll
          for (int e = 0; e < 16; ++e) sc[qb][e] -= d;
        }
        float psum = 0.0f;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float p = __builtin_amdgcn_exp2f(sc[qb][e]);
          if constexpr (!C::MFMA_SUM) psum = e ? psum + p : p;   // no add of 0 to start
          pb[qb][e >> 3][e & 7] = (bf16)p;
        }
        if constexpr (!C::MFMA_SUM) l_part[qb] += psum;
      }
    };
    auto pv = [&](bf16x8 (*va)[C::HB], bf16x8 (*pb)[2]) {
#pragma unroll
      for (int ch = 0; ch < 2; ++ch)
#pragma unroll
        for (int hb = 0; hb < C::HB; ++hb)
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            o[qb][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[ch][hb], pb[qb][ch], o[qb][hb], 0, 0, 0);
    };
    // the same with each 16-key chunk's V^T fragments read right before its MFMAs
    auto pv_direct = [&](int kb, bf16x8 (*pb)[2]) {
#pragma unroll
      for (int ch = 0; ch < 2; ++ch)
#pragma unroll
        for (int hb = 0; hb < C::HB; ++hb) {
          union { bf16x8 v; v4i16 h[2]; } u;
#pragma unroll
          for (int half = 0; half < 2; ++half) {
            const int rbase = (kb * 32 + 16 * ch + 8 * half) * C::R * 16;
            u.h[half] = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (lds_v4i16*)(lds + buf * C::BUF + C::TILE + rbase + vofs[hb]));
          }
          const bf16x8 vv = (hb == C::HB - 1 && pad_lane) ? ones : u.v;
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            o[qb][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vv, pb[qb][ch], o[qb][hb], 0, 0, 0);
        }
    };

    bf16x8 va[2][C::HB], pa[QB][2];
    if constexpr (C::OVERLAP) {
      f32x16 sa[QB], sb[QB];
      scores(0, sa);
      if (nkb == 2) scores(1, sb);
      read_v(0, va);
      __builtin_amdgcn_sched_barrier(0);
      softmax(0, t == 0, sa, pa);
      pv(va, pa);
      if (nkb == 2) {
        __builtin_amdgcn_sched_barrier(0);
        read_v(1, va);
        softmax(1, false, sb, pa);
        pv(va, pa);
      }
    } else {
      // one half's scores live at a time
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        if (kb >= nkb) break;
        f32x16 sc[QB];
        scores(kb, sc);
        if constexpr (C::V_DIRECT) {
          softmax(kb, t == 0 && kb == 0, sc, pa);
          pv_direct(kb, pa);
        } else {
          read_v(kb, va);
          softmax(kb, t == 0 && kb == 0, sc, pa);
          pv(va, pa);
        }
      }
    }
  }

  // Every wave is past the last tile (its reads done): the two K / V buffers now
  // hold each wave's 32 x HD output block, row-major with the 16-byte chunks of
  // row r rotated by r, so the stores leave as whole rows (8 rows of a 64-dim
  // head per instruction) instead of 16-byte pieces of 32 rows.
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __syncthreads();
  if (!active) return;
  constexpr int NCH = HD / 8;   // 16-byte chunks per output row
  static_assert(C::NW * QB * 32 * HD * 2 <= 2 * C::BUF && (32 * NCH) % 64 == 0, "output staging");
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    char* stg = smem + (wave * QB + qb) * 32 * HD * 2;
    const float inv = C::MFMA_SUM ? 1.0f / o[qb][C::HB - 1][8]
                                  : 1.0f / (l_part[qb] + __shfl_xor(l_part[qb], 32, 64));
#pragma unroll
    for (int hb = 0; hb < C::HB; ++hb)
#pragma unroll
      for (int e4 = 0; e4 < 4; ++e4) {
        const int d = hb * 32 + e4 * 8 + g * 4;   // lanes g = 0, 1 hold the two halves of chunk d / 8
        if (d < HD) {
          union { uint2 u; bf16 h[4]; } st;
#pragma unroll
          for (int e = 0; e < 4; ++e) st.h[e] = (bf16)(o[qb][hb][e4 * 4 + e] * inv);
          *reinterpret_cast<uint2*>(stg + l32 * HD * 2 + (((d >> 3) + l32) % NCH) * 16 + g * 8) = st.u;
        }
      }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // the wave's own writes are visible to it
    const int qb0 = qw0 + qb * 32;
#pragma unroll
    for (int k = 0; k < 32 * NCH / 64; ++k) {
      const int c = lane + 64 * k, row = c / NCH, ch = c % NCH;
      const uint4 val = *reinterpret_cast<const uint4*>(stg + row * HD * 2 + ((ch + row) % NCH) * 16);
      if (qb0 + row < s1)
        *reinterpret_cast<uint4*>(static_cast<bf16*>(a.out) + (long)(qb0 + row) * a.ldo + h * HD + ch * 8) = val;
    }
  }
}

template <int HD, int QB, int QT>
hipError_t launch_hd(const AttnArgs& a, const AttnWork& w, int total_tiles, hipStream_t s) {
  using C = AttnCfg<HD, QB, QT>;
  constexpr int lds = 2 * C::BUF;
  hipLaunchKernelGGL((attn_bf16_dma_kernel<HD, QB, QT>), dim3((unsigned)(total_tiles * a.heads)), dim3(64 * C::NW), lds,
                     s, a, w);
  return hipGetLastError();
}

}  // namespace

// 256-query tiles for head_dim 80 when they add at most 2% query slots over
// 128-query tiles (video clips: none; batches of 32 mixed-size images: 1-2%):
// on equal slots they measured 4-6% faster (8192-token clips), 3.6% more
// slots (3600-token images) still 0.5-2.4% faster; for head_dim 64 (577- and
// 1500-token rows) they measured no faster or slower.
// Each query's arithmetic does not depend on the tile that holds it, so the
// choice never changes a result.
int attention_dma_q_tile(int hd, const int* cu, int n) {
  if (hd != 80) return 128;
  long s128 = 0, s256 = 0;
  for (int r = 0; r < n; ++r) {
    const long L = cu[r + 1] - cu[r];
    s128 += (L + 127) / 128 * 128;
    s256 += (L + 255) / 256 * 256;
  }
  return s256 * 100 <= s128 * 102 ? 256 : 128;
}

bool attention_dma_supported(const AttnArgs& a, int N) {
  return (a.hd == 64 || a.hd == 80) && a.ldqkv % 8 == 0 && (uintptr_t)a.qkv % 16 == 0 &&
         (double)N * a.ldqkv * 2 < 4294967296.0;
}

hipError_t launch_attention_bf16_dma(const AttnArgs& a, const AttnWork& w, int total_tiles, hipStream_t s,
                                     const char** kname) {
  if (w.qt == 256 && a.hd == 80) { *kname = "attn_bf16_hd80_q256"; return launch_hd<80, 1, 256>(a, w, total_tiles, s); }
  if (w.qt != 128) return hipErrorInvalidValue;
  if (a.hd == 64) { *kname = "attn_bf16_hd64"; return launch_hd<64, 1, 128>(a, w, total_tiles, s); }
  if (a.hd == 80) { *kname = "attn_bf16_hd80"; return launch_hd<80, 1, 128>(a, w, total_tiles, s); }
  return hipErrorInvalidValue;
}

}  // namespace eas

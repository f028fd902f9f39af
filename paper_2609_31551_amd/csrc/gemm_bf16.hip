// bf16 MFMA GEMM for the encoder's dense projections (QKV, attention output,
// MLP, merger, audio front end).  C[m, n] = sum_k A[m, k] * B[n, k]: both
// operands K-contiguous ("NT"), the natural layout of activations
// [tokens, in] and of Linear weights [out, in].
//
// Design (gfx950, one workgroup per BM x BN output tile):
//  * Operands reach LDS by direct DMA: global_load_lds_dwordx4 moves 16 bytes
//    per lane from HBM/L2 into LDS without passing through VGPRs.  With a
//    64-wide k-step one wave instruction fills 1 KB = 8 rows x 128 bytes, so
//    every lane group reads whole 128-byte lines.  The lane -> (row, 16-byte
//    chunk) assignment applies an XOR swizzle (chunk ^ ((row >> 1) & 7)) that
//    spreads the MFMA operand reads -- 32 rows at one k offset, 16 lanes per
//    LDS cycle over 64 banks -- without conflicts.
//  * ST LDS stages of 64 k (two for full launches, three for the small-tile
//    path of latency-bound ones): tile k+ST-1 streams in while tile k is
//    consumed.  The DMA is issued from inline assembly so the compiler does
//    not serialise it against the LDS reads; completion is tracked with
//    explicit s_waitcnt vmcnt and one workgroup barrier per k-step.
//  * v_mfma_f32_32x32x16_bf16, each wave a (BM/WGM) x (BN/WGN) sub-tile of
//    32 x 32 blocks (16 waves of 64 x 64 for the 256 x 256 tile: four waves
//    per SIMD keep more stores in flight in the epilogue); operand
//    fragments for the next 16-wide k slice are read while the current
//    slice's MFMAs run (the issue order is pinned: one read between two
//    MFMAs), and the barrier sits before the last slice so its wait overlaps
//    queued MFMAs.
//  * Tiles are handed out XCD-aware: workgroups are dispatched round-robin
//    over the 8 XCDs, so block b is remapped to give every XCD a contiguous
//    run of output tiles, ordered in groups of 4 tile rows swept column by
//    column, so the tiles an XCD runs together share operand panels in its L2.
//  * Fused epilogue through LDS: each wave stages 32 rows of its fp32
//    accumulators, then every lane owns 8 consecutive columns of a row and
//    applies bias, GELU / QuickGELU, a position-table row and the fp32
//    residual before one 16-byte (bf16) or 2 x 16-byte (fp32) store.
//  * Bias / activation epilogues with up to 2048-wide k, and fp32 residual
//    epilogues (O-projection, FC2) of any k, run a persistent variant (below)
//    whose epilogue stores keep draining while the next tile's k-loop runs.
//  * Every output element accumulates k in the same order (16-wide MFMA
//    slices, ascending) whatever the kernel, tile shape or M, so a
//    request's result does not depend on what else is in the micro-batch.
#include "common.h"

namespace eas {
namespace {

constexpr int BK = 64;
constexpr int kResAhead = 1;
constexpr int kStoreNT = 2;    // buffer-store cache policy: non-temporal (NT bit)
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// M0 carries the LDS base of each DMA; nothing else in these kernels uses M0
// (checked in the generated code), so setting it here cannot disturb the
// compiler's own code even though it treats M0 as reserved.
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(unsigned lds_addr, unsigned voff, const void* gbase) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2\n"
               :: "s"(lds_addr), "v"(voff), "s"(gbase) : "memory", "m0");
}
template <int N> __device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}
__device__ __forceinline__ void wait_lds() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

template <int BM, int BN, int WGM, int WGN, int ST = 2>
struct Cfg {
  static constexpr int NW = WGM * WGN, NT = 64 * NW;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int TA = BM * BK * 2, TB = BN * BK * 2, STAGE = TA + TB;
  static constexpr int RPI = 1024 / (BK * 2);                   // rows per DMA instruction
  static constexpr int CPR = BK / 8;                            // 16-byte chunks per row
  static constexpr int DA = BM / RPI / NW, DB = BN / RPI / NW;   // DMA instructions per wave per stage
  static constexpr int DPS = DA + DB;
  static constexpr int SLD = WN + 4;                            // epilogue slab row (floats)
  static constexpr int LDS = ST * STAGE > NW * 32 * SLD * 4 ? ST * STAGE : NW * 32 * SLD * 4;
  static_assert(BM % (RPI * NW) == 0 && BN % (RPI * NW) == 0, "DMA split");
  static_assert(DPS * (ST - 1) < 64, "vmcnt range");
  // conflict-free chunk swizzle for 128-byte rows: 16 rows per LDS cycle hit 16 distinct 16-byte slots
  __device__ static int sw(int row) { return (row >> 1) & 7; }
};

// XCD-aware block -> tile index (bijective on [0, nb)).
__device__ __forceinline__ int xcd_tile(int b, int nb) {
  const int per = (nb + 7) / 8, x = b % 8, s = b / 8;
  const int full = nb % 8 == 0 ? 8 : nb % 8;   // XCDs that receive `per` blocks
  return (x < full ? x * per : full * per + (x - full) * (per - 1)) + s;
}

// Linear tile index -> (tile row, tile column), in groups of GROUP_M tile rows
// swept column by column, so the ~32 tiles an XCD runs at once form a
// GROUP_M x 8 block and share fewer operand panels in its L2.
constexpr int GROUP_M = 4;
__device__ __forceinline__ void tile_coords(int t, int mt, int nt, int& mi, int& ni) {
  const int g = t / (GROUP_M * nt), r = t % (GROUP_M * nt);
  const int rows = min(GROUP_M, mt - g * GROUP_M);
  ni = r / rows;
  mi = g * GROUP_M + r % rows;
}

// Waits until at most n k-tiles' DMA (of DPS instructions each) are in flight, 0 <= n <= N.
template <int DPS, int N>
__device__ __forceinline__ void wait_tiles(int n) {
  if constexpr (N > 0) {
    if (n >= N) { wait_vm<N * DPS>(); return; }
    wait_tiles<DPS, N - 1>(n);
  } else {
    wait_vm<0>();
  }
}

template <int BM, int BN, int WGM, int WGN, int ST>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_tile_kernel(GemmArgs a) {
  using C = Cfg<BM, BN, WGM, WGN, ST>;
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const unsigned lds0 = (unsigned)(size_t)((__attribute__((address_space(3))) char*)smem);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int tiles_n = (a.N + BN - 1) / BN;
  int mi, ni;
  tile_coords(xcd_tile(blockIdx.x, gridDim.x), (a.M + BM - 1) / BM, tiles_n, mi, ni);
  const int m0 = mi * BM, n0 = ni * BN;
  const int KT = a.K / BK;
  const bf16* A = static_cast<const bf16*>(a.A);
  const bf16* B = static_cast<const bf16*>(a.B);

  // DMA sources: instruction j of this wave fills tile rows (wave*D + j)*8 .. +8;
  // lane i -> row +i/8, physical chunk i%8 holding logical chunk (i%8) ^ sw(row).
  // Rows past M or N re-read the last row; their results are never stored.
  unsigned a_off[C::DA], b_off[C::DB];
  {
    const int rr = lane / C::CPR, pch = lane % C::CPR;
#pragma unroll
    for (int j = 0; j < C::DA; ++j) {
      const int r = (wave * C::DA + j) * C::RPI + rr;
      const int gm = min(m0 + r, a.M - 1);
      a_off[j] = (unsigned)(((long)gm * a.lda + (pch ^ C::sw(r)) * 8) * 2);
    }
#pragma unroll
    for (int j = 0; j < C::DB; ++j) {
      const int r = (wave * C::DB + j) * C::RPI + rr;
      int gn = min(n0 + r, a.N - 1);
      if (a.rope_pos) gn = rope_src_row(gn, a.rope_hd, a.rope_hd_inv, a.rope_cols);
      b_off[j] = (unsigned)(((long)gn * a.ldb + (pch ^ C::sw(r)) * 8) * 2);
    }
  }
  auto issue = [&](int kt, int st) {
    const unsigned base = lds0 + st * C::STAGE;
    const bf16* ga = A + kt * BK;
    const bf16* gb = B + kt * BK;
#pragma unroll
    for (int j = 0; j < C::DA; ++j) dma16(base + (wave * C::DA + j) * 1024, a_off[j], ga);
#pragma unroll
    for (int j = 0; j < C::DB; ++j) dma16(base + C::TA + (wave * C::DB + j) * 1024, b_off[j], gb);
  };

  // operand fragment reads: row wm*WM + i*32 + lane%32, logical chunk 2*slice + lane/32;
  // the swizzle only depends on the row's low bits, i.e. on lane%32
  const int lrow = lane & 31, g = lane >> 5, swz = C::sw(lrow);
  const int a_row = (wm * C::WM + lrow) * BK * 2, b_row = (wn * C::WN + lrow) * BK * 2;
  constexpr int NH = BK / 16;   // 16-wide k slices per k-step
  int cofs[NH];
#pragma unroll
  for (int h = 0; h < NH; ++h) cofs[h] = ((2 * h + g) ^ swz) << 4;
  f32x16 acc[C::FM][C::FN];
#pragma unroll
  for (int i = 0; i < C::FM; ++i)
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  bf16x8 fa[2][C::FM], fb[2][C::FN];
  auto load_frags = [&](int st, int cofs, bf16x8* fa, bf16x8* fb) {
    const char* As = smem + st * C::STAGE;
    const char* Bs = As + C::TA;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) fa[i] = *reinterpret_cast<const bf16x8*>(As + a_row + i * 32 * BK * 2 + cofs);
#pragma unroll
    for (int j = 0; j < C::FN; ++j) fb[j] = *reinterpret_cast<const bf16x8*>(Bs + b_row + j * 32 * BK * 2 + cofs);
  };
  auto mma = [&](const bf16x8* fa, const bf16x8* fb) {
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[i], fb[j], acc[i][j], 0, 0, 0);
  };
  // pin the issue order of one slice: each fragment read of the next slice
  // goes between two MFMAs of this one, so LDS latency hides under the MFMAs
  auto interleave = [&]() {
    constexpr int NR = C::FM + C::FN, NM = C::FM * C::FN, NP = NR < NM ? NR : NM;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
    }
    if constexpr (NM > NP) __builtin_amdgcn_sched_group_barrier(0x008, NM - NP, 0);
    if constexpr (NR > NP) __builtin_amdgcn_sched_group_barrier(0x100, NR - NP, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  // prologue: tiles 0 .. ST-1 in flight; wait for tile 0
#pragma unroll
  for (int s = 0; s < ST; ++s)
    if (s < KT) issue(s, s);
  wait_tiles<C::DPS, ST - 1>(min(ST, KT) - 1);
  __syncthreads();
  load_frags(0, cofs[0], fa[0], fb[0]);

  // every k-tile but the last; the loop body has no branch around its MFMAs,
  // so the next tile's first fragment reads interleave with this tile's last slice
  for (int kt = 0; kt < KT - 1; ++kt) {
    const int st = kt % ST;
#pragma unroll
    for (int h = 0; h < NH - 1; ++h) {
      load_frags(st, cofs[h + 1], fa[(h + 1) & 1], fb[(h + 1) & 1]);
      mma(fa[h & 1], fb[h & 1]);
      interleave();
    }
    // this wave's reads of stage st are done once lgkmcnt drains; tile kt+1
    // has landed once only the tiles after it (up to kt+ST-1) are in flight;
    // after the barrier every wave is past stage st, refilled with tile kt+ST
    wait_lds();
    wait_tiles<C::DPS, ST - 2>(min(ST - 2, KT - 2 - kt));
    __builtin_amdgcn_s_barrier();
    if (kt + ST < KT) issue(kt + ST, st);
    __builtin_amdgcn_sched_barrier(0);
    load_frags((kt + 1) % ST, cofs[0], fa[NH & 1], fb[NH & 1]);
    mma(fa[(NH - 1) & 1], fb[(NH - 1) & 1]);
    interleave();
  }
  {
    const int st = (KT - 1) % ST;
#pragma unroll
    for (int h = 0; h < NH - 1; ++h) {
      load_frags(st, cofs[h + 1], fa[(h + 1) & 1], fb[(h + 1) & 1]);
      mma(fa[h & 1], fb[h & 1]);
      interleave();
    }
    mma(fa[(NH - 1) & 1], fb[(NH - 1) & 1]);
  }

  // ---- fused epilogue: per wave, 32-row slabs of its WM x WN sub-tile through LDS ----
  wait_lds();
  __builtin_amdgcn_s_barrier();
  float* slab = reinterpret_cast<float*>(smem) + wave * 32 * C::SLD;
  constexpr int LPR = C::WN / 8;   // lanes per row, 8 columns each
  constexpr int RPP = 64 / LPR;    // rows per pass
  const int prow = lane / LPR, pc = (lane % LPR) * 8;
  const int n = n0 + wn * C::WN + pc;
  const bool nok = n < a.N;        // N % 8 == 0: a lane's 8 columns are all in or all out
  float bv[8];
  {
    const bf16* bias = static_cast<const bf16*>(a.bias);
#pragma unroll
    for (int e = 0; e < 8; ++e) bv[e] = (bias && nok) ? (float)bias[n + e] : 0.0f;
  }
  const int act = a.act;
#pragma unroll
  for (int i = 0; i < C::FM; ++i) {
#pragma unroll
    for (int j = 0; j < C::FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        slab[((e >> 2) * 8 + g * 4 + (e & 3)) * C::SLD + j * 32 + lrow] = acc[i][j][e];
    wait_lds();
    __builtin_amdgcn_wave_barrier();
    const int mrow0 = m0 + wm * C::WM + i * 32;
#pragma unroll 2
    for (int p = 0; p < 32 / RPP; ++p) {
      const int r = p * RPP + prow, m = mrow0 + r;
      if (m < a.M && nok) {
        const float4 s0 = *reinterpret_cast<const float4*>(slab + r * C::SLD + pc);
        const float4 s1 = *reinterpret_cast<const float4*>(slab + r * C::SLD + pc + 4);
        float v[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += bv[e];
        if (act == ACT_GELU) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = gelu_erf(v[e]);
        } else if (act == ACT_QUICKGELU) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = quick_gelu(v[e]);
        }
        if (a.rope_pos && n < a.rope_cols) {   // four interleaved pairs, slots i0 .. i0 + 3
          const int4 rp = a.rope_pos[m];
          const int i0 = rope_in_head(n, a.rope_hd, a.rope_hd_inv) >> 1;
#pragma unroll
          for (int t = 0; t < 4; ++t) rope_rotate(v[2 * t], v[2 * t + 1], rope_turns(a, i0 + t, rp.x, rp.y, rp.z));
        }
        if (a.pos) {
          const int pr = a.pos_idx ? a.pos_idx[m] : m % a.pos_period;
          const long pi = (long)pr * a.ld_pos + n;
          if (a.pos_f32) {
            const float4 p0 = *reinterpret_cast<const float4*>(static_cast<const float*>(a.pos) + pi);
            const float4 p1 = *reinterpret_cast<const float4*>(static_cast<const float*>(a.pos) + pi + 4);
            v[0] += p0.x; v[1] += p0.y; v[2] += p0.z; v[3] += p0.w;
            v[4] += p1.x; v[5] += p1.y; v[6] += p1.z; v[7] += p1.w;
          } else {
            union { uint4 u; bf16 h[8]; } pb;
            pb.u = *reinterpret_cast<const uint4*>(static_cast<const bf16*>(a.pos) + pi);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] += (float)pb.h[e];
          }
        }
        if (a.resid) {
          const float4 r0 = *reinterpret_cast<const float4*>(a.resid + (long)m * a.ldr + n);
          const float4 r1 = *reinterpret_cast<const float4*>(a.resid + (long)m * a.ldr + n + 4);
          v[0] += r0.x; v[1] += r0.y; v[2] += r0.z; v[3] += r0.w;
          v[4] += r1.x; v[5] += r1.y; v[6] += r1.z; v[7] += r1.w;
        }
        const long oi = (long)m * a.ldo + n;
        if (a.out_f32) {
          float* o = static_cast<float*>(a.out) + oi;
          *reinterpret_cast<float4*>(o) = make_float4(v[0], v[1], v[2], v[3]);
          *reinterpret_cast<float4*>(o + 4) = make_float4(v[4], v[5], v[6], v[7]);
        } else {
          union { uint4 u; bf16 h[8]; } pk;
#pragma unroll
          for (int e = 0; e < 8; ++e) pk.h[e] = (bf16)v[e];
          *reinterpret_cast<uint4*>(static_cast<bf16*>(a.out) + oi) = pk.u;
        }
      }
    }
    wait_lds();
    __builtin_amdgcn_wave_barrier();
  }
}

// ---- persistent variant with an asynchronous epilogue (bias, activation, fp32 residual) ----
//
// A fixed grid of workgroups walks the tile list (block b takes tiles b, b + grid,
// ...; the same XCD-aware order as above), so a CU moves to its next tile
// without a relaunch: that tile's k-tile 0 streams in under the last k-step and
// its k-tile 1 right after the epilogue.  The epilogue issues no load the compiler
// knows of -- the bias row reaches LDS by DMA with the operands -- and writes
// through buffer stores whose count per wave is fixed (lanes outside the
// output get an out-of-range offset and are dropped by the buffer unit), so the
// next tile's waits can count past them: vector memory operations complete in
// issue order, and the stores keep draining while the next tile's k-loop runs.
// The MFMA operands are swapped (C^T blocks: each lane holds 4 consecutive
// columns of one row): with bf16 output the bias and activation are applied in
// registers and a finished 32-row block row is staged with 8-byte writes in the
// LDS stage the last k-tile used (free until the next tile's k-tile 1), so
// each store instruction writes whole 128-byte rows (+1% against 64-byte half
// rows through a 2 KB per-wave slab); fp32 sums go through a 4 KB slab with
// 16-byte writes and leave, like the fp32 residual they add, in instructions of
// 8 whole 128-byte rows (1-3% against 16 rows of scattered 16-byte pieces).  The products, their order over k and the
// per-element epilogue arithmetic are the same as in the kernel above, so the
// two kernels give identical bits.
template <int BM, int BN, int WGM, int WGN, int OUTF32>
struct ACfg : Cfg<BM, BN, WGM, WGN> {
  // per-wave epilogue slab: a 32 x 32 block of fp32 sums, or of finished bf16
  // outputs (bias and activation applied in registers first)
  static constexpr int SLAB = 32 * 32 * (OUTF32 ? 4 : 2);
  static constexpr int LDS = 2 * Cfg<BM, BN, WGM, WGN>::STAGE + Cfg<BM, BN, WGM, WGN>::NW * SLAB;
  static_assert(Cfg<BM, BN, WGM, WGN>::WN <= 512 && 1024 <= SLAB, "bias row fits one DMA and the slab");
  __device__ static int sw16(int row) { return (row >> 2) & 3; }   // 16-byte chunk swizzle of 64-byte rows
};

template <int BM, int BN, int WGM, int WGN, int OUTF32, int RES = 0, int ROPE = 0>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_async_kernel(GemmArgs a, int n_tiles) {
  using C = ACfg<BM, BN, WGM, WGN, OUTF32>;
  constexpr int S = C::FM * C::FN * 2 * (OUTF32 ? 2 : 1);   // buffer stores per wave per tile
  constexpr int L = RES ? C::FM * C::FN * 4 : 0;              // residual loads per wave per tile
  constexpr int E = 1 + ROPE;                                 // epilogue DMAs per wave per tile (bias, positions)
  static_assert(C::DPS + S + E < 64, "vmcnt range");
  static_assert(!RES || OUTF32, "the residual stream is fp32");
  static_assert(!ROPE || (!OUTF32 && C::WM == 64 && C::SLAB >= 2048), "rotary epilogue: bf16 output, 64-row waves");
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const unsigned lds0 = (unsigned)(size_t)((__attribute__((address_space(3))) char*)smem);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.N + BN - 1) / BN;
  const int KT = a.K / BK;   // >= 2
  const bf16* A = static_cast<const bf16*>(a.A);
  const bf16* B = static_cast<const bf16*>(a.B);
  const bf16* bias = a.bias ? static_cast<const bf16*>(a.bias) : B;
  const float bias_on = a.bias ? 1.0f : 0.0f;
  const int rr = lane / C::CPR, pch = lane % C::CPR;
  unsigned a_off[C::DA], b_off[C::DB];
  auto set_offsets = [&](int m0, int n0) {
#pragma unroll
    for (int j = 0; j < C::DA; ++j) {
      const int r = (wave * C::DA + j) * C::RPI + rr;
      a_off[j] = (unsigned)(((long)min(m0 + r, a.M - 1) * a.lda + (pch ^ C::sw(r)) * 8) * 2);
    }
#pragma unroll
    for (int j = 0; j < C::DB; ++j) {
      const int r = (wave * C::DB + j) * C::RPI + rr;
      int gn = min(n0 + r, a.N - 1);
      if constexpr (ROPE) gn = rope_src_row(gn, a.rope_hd, a.rope_hd_inv, a.rope_cols);
      b_off[j] = (unsigned)(((long)gn * a.ldb + (pch ^ C::sw(r)) * 8) * 2);
    }
  };
  auto issue = [&](int kt, int st) {
    const unsigned base = lds0 + st * C::STAGE;
#pragma unroll
    for (int j = 0; j < C::DA; ++j) dma16(base + (wave * C::DA + j) * 1024, a_off[j], A + kt * BK);
#pragma unroll
    for (int j = 0; j < C::DB; ++j) dma16(base + C::TA + (wave * C::DB + j) * 1024, b_off[j], B + kt * BK);
  };
  auto tile_of = [&](int t, int& m0, int& n0) {
    int mi, ni;
    tile_coords(xcd_tile(t, n_tiles), tiles_m, tiles_n, mi, ni);
    m0 = mi * BM;
    n0 = ni * BN;
  };
  const unsigned slab_lds = lds0 + 2 * C::STAGE + wave * C::SLAB;
  char* slab_b = smem + 2 * C::STAGE + wave * C::SLAB;
  float* slab = reinterpret_cast<float*>(slab_b);
  // this wave's WN bias values -> slab bytes [0, 2 WN); the other lanes repeat them
  // with the rotary epilogue, the (t, h, w) positions of the wave's 64 rows -> slab bytes [1024, 2048)
  auto issue_bias = [&](int n0, int m0) {
    const int n = a.bias ? min(n0 + wn * C::WN + (lane % (C::WN / 8)) * 8, a.N - 8) : 0;
    dma16(slab_lds, (unsigned)(n * 2), bias);
    if constexpr (ROPE) dma16(slab_lds + 1024, (unsigned)(min(m0 + wm * C::WM + lane, a.M - 1) * 16), a.rope_pos);
  };

  const int lrow = lane & 31, g = lane >> 5, swz = C::sw(lrow);
  const int a_row = (wm * C::WM + lrow) * BK * 2, b_row = (wn * C::WN + lrow) * BK * 2;
  constexpr int NH = BK / 16;
  int cofs[NH];
#pragma unroll
  for (int h = 0; h < NH; ++h) cofs[h] = ((2 * h + g) ^ swz) << 4;
  f32x16 acc[C::FM][C::FN];
  bf16x8 fa[2][C::FM], fb[2][C::FN];
  auto load_frags = [&](int st, int cofs, bf16x8* fa, bf16x8* fb) {
    const char* As = smem + st * C::STAGE;
    const char* Bs = As + C::TA;
#pragma unroll
    for (int i = 0; i < C::FM; ++i) fa[i] = *reinterpret_cast<const bf16x8*>(As + a_row + i * 32 * BK * 2 + cofs);
#pragma unroll
    for (int j = 0; j < C::FN; ++j) fb[j] = *reinterpret_cast<const bf16x8*>(Bs + b_row + j * 32 * BK * 2 + cofs);
  };
  auto mma = [&](const bf16x8* fa, const bf16x8* fb) {
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
  };
  auto interleave = [&]() {
    constexpr int NR = C::FM + C::FN, NM = C::FM * C::FN;
    static_assert(NM >= NR, "more reads than MFMAs per slice");
#pragma unroll
    for (int i = 0; i < NR; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NM - NR, 0);
    __builtin_amdgcn_sched_barrier(0);
  };
  const int es = OUTF32 ? 4 : 2;
  const int act = a.act;

  int t = blockIdx.x, m0, n0;
  tile_of(t, m0, n0);
  set_offsets(m0, n0);
  issue(0, 0);
  issue(1, 1);
  int sb = 0;          // stage of this tile's k-tile 0
  bool first = true;
  for (;;) {
    const int tn = t + gridDim.x;
    const bool has_next = tn < n_tiles;
    int m0n = 0, n0n = 0;
    if (has_next) tile_of(tn, m0n, n0n);
    // k-tile 0: issued ahead of k-tile 1 and of the previous tile's S stores (with a
    // residual: ahead of the previous epilogue's L loads and S stores, then k-tile 1;
    // a count past vmcnt's range waits for a few loads that have completed anyway)
    if (first) wait_vm<C::DPS>();
    else if constexpr (RES) wait_vm<(C::DPS + L + S < 63 ? C::DPS + L + S : 63)>();
    else wait_vm<C::DPS + S>();
    __builtin_amdgcn_s_barrier();
    issue_bias(n0, m0);
#pragma unroll
    for (int i = 0; i < C::FM; ++i)
#pragma unroll
      for (int j = 0; j < C::FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
    load_frags(sb, cofs[0], fa[0], fb[0]);
    for (int kt = 0; kt < KT - 1; ++kt) {
      const int st = (sb + kt) & 1;
#pragma unroll
      for (int h = 0; h < NH - 1; ++h) {
        load_frags(st, cofs[h + 1], fa[(h + 1) & 1], fb[(h + 1) & 1]);
        mma(fa[h & 1], fb[h & 1]);
        interleave();
      }
      wait_lds();
      // k-tile kt+1 has landed; at kt == 0 the previous stores and the bias DMA may follow it
      // (with a residual, k-tile 1 follows the previous epilogue: only the bias DMA)
      if (kt == 0) {
        if (first || RES || !OUTF32) wait_vm<E>();
        else wait_vm<S + E>();
      } else {
        wait_vm<0>();
      }
      __builtin_amdgcn_s_barrier();
      if (kt + 2 < KT) {
        issue(kt + 2, st);
      } else if (has_next) {
        set_offsets(m0n, n0n);
        issue(0, st);
      }
      __builtin_amdgcn_sched_barrier(0);
      load_frags(st ^ 1, cofs[0], fa[NH & 1], fb[NH & 1]);
      mma(fa[(NH - 1) & 1], fb[(NH - 1) & 1]);
      interleave();
    }
    // fp32 epilogue: eight lanes cover a 128-byte row of a 32 x 32 block, 4 columns
    // each, so every load and store instruction moves 8 whole rows; four 8-row
    // passes per block.  Residual epilogue: a block's 4 loads are issued up to
    // kResAhead blocks ahead (the first block's under the last k-step).  The loads
    // are ordinary buffer loads, so the compiler waits for them itself: no DMA is
    // issued between them and their use, so its counts are exact.  Rows past M and
    // columns past N read 0.
    const int prow = lane >> 3, pc = (lane & 7) * 4;
    const int rows = min(BM, a.M - m0);
    constexpr int NB = C::FM * C::FN, RR = kResAhead + 1;
    u32x4 rq[RR][4];   // [block % RR][pass]
    __amdgpu_buffer_rsrc_t res_rsrc;
    if constexpr (RES)
      res_rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(a.resid) + (size_t)m0 * a.ldr, 0,
                                                   rows * a.ldr * 4, 0x00020000);
    auto rload = [&](int b, u32x4 (&r)[4]) {
      const int i = b / C::FN, j = b % C::FN;
      const int n = n0 + wn * C::WN + j * 32 + pc;
      // bit 31 set for columns past N (the sign of N - 1 - n), without a select,
      // which the compiler would turn into a branch around each load; the row step
      // of a pass is a scalar added to one per-block offset
      const unsigned off0 = (unsigned)(((wm * C::WM + i * 32 + prow) * a.ldr + n) * 4) |
                            ((unsigned)(a.N - 1 - n) & 0x80000000u);
#pragma unroll
      for (int p = 0; p < 4; ++p)
        r[p] = __builtin_amdgcn_raw_buffer_load_b128(res_rsrc, off0 + (unsigned)(p * 8 * a.ldr * 4), 0, 0);
    };
    {
      const int st = (sb + KT - 1) & 1;
      if constexpr (RES) rload(0, rq[0]);
#pragma unroll
      for (int h = 0; h < NH - 1; ++h) {
        load_frags(st, cofs[h + 1], fa[(h + 1) & 1], fb[(h + 1) & 1]);
        mma(fa[(h) & 1], fb[(h) & 1]);
        interleave();
      }
      mma(fa[(NH - 1) & 1], fb[(NH - 1) & 1]);
    }
    wait_lds();
    // the bias has landed: with KT > 2 the wait of k-step 1 covered it; with KT == 2
    // only the next tile's k-tile 0 (and the first residual loads) were issued after it
    if (KT == 2) {
      if (has_next) wait_vm<C::DPS + L / (C::FM * C::FN)>();
      else wait_vm<L / (C::FM * C::FN)>();
    }
    __builtin_amdgcn_s_barrier();   // every wave is past the last stage
    if (!RES && OUTF32 && has_next) issue(1, (sb + KT + 1) & 1);
    __builtin_amdgcn_sched_barrier(0);

    // ---- epilogue: one 32 x 32 block at a time through the wave's slab ----
    const __amdgpu_buffer_rsrc_t out_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        static_cast<char*>(a.out) + (size_t)m0 * a.ldo * es, 0, rows * a.ldo * es, 0x00020000);
    if constexpr (!OUTF32) {
      // bf16 output: bias and activation on the sums in place (columns 8q + 4g + e
      // of each block), then the finished 32 x 32 bf16 block goes through the slab
      // the stage the last k-tile used is free until the next tile's k-tile 1 (DMA'd
      // after the epilogue): each wave stages a 32 x WN block row there, row-major
      // with the 16-byte chunks of row r swizzled by r & 7, and stores whole rows
      constexpr int RS = C::WN * 2, CPRS = C::WN / 8;
      static_assert(C::NW * 32 * RS <= C::STAGE && (32 * CPRS) % 64 == 0, "bf16 output staging");
      char* stg = smem + ((sb + KT - 1) & 1) * C::STAGE + wave * 32 * RS;
      // read-back: lane -> row r0 (+ RST per pass), 16-byte chunk ch; the row's swizzle
      // r & 7 is r0 & 7 on passes with (k * RST) % 8 == 0 (rd0), else (r0 + RST) & 7 (rd1)
      constexpr int RST = 64 / CPRS;
      static_assert(RST == 4 || RST == 8, "rows per read-back pass");
      const int r0 = lane / CPRS, ch = lane % CPRS;
      const int rd0 = r0 * RS + ((ch ^ (r0 & 7)) << 4);
      const int rd1 = r0 * RS + ((ch ^ ((r0 + RST) & 7)) << 4);
      const int nst = n0 + wn * C::WN + ch * 8;
      const unsigned st0 = nst < a.N ? (unsigned)(((wm * C::WM + r0) * a.ldo + nst) * 2) : 0x80000000u;
#pragma unroll
      for (int i = 0; i < C::FM; ++i) {
        int pt = 0, ph = 0, pw = 0;   // the lane's row position in block row i
        if constexpr (ROPE) {
          const int4 p = *reinterpret_cast<const int4*>(slab_b + 1024 + (i * 32 + lrow) * 16);
          pt = p.x;
          ph = p.y;
          pw = p.z;
        }
#pragma unroll
        for (int j = 0; j < C::FN; ++j) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            union { uint2 u; bf16 h[4]; } bb, pk;
            bb.u = *reinterpret_cast<const uint2*>(slab_b + (j * 32 + 8 * q + 4 * g) * 2);
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = acc[i][j][4 * q + e] + (float)bb.h[e] * bias_on;
            if (act == ACT_GELU) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = gelu_erf(v[e]);
            } else if (act == ACT_QUICKGELU) {
#pragma unroll
              for (int e = 0; e < 4; ++e) v[e] = quick_gelu(v[e]);
            }
            if constexpr (ROPE) {   // two interleaved pairs: columns 8q + 4g + (0, 1) and (2, 3)
              const int n = n0 + wn * C::WN + j * 32 + 8 * q + 4 * g;
              if (n < a.rope_cols) {
                const int i0 = rope_in_head(n, a.rope_hd, a.rope_hd_inv) >> 1;
                rope_rotate(v[0], v[1], rope_turns(a, i0, pt, ph, pw));
                rope_rotate(v[2], v[3], rope_turns(a, i0 + 1, pt, ph, pw));
              }
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) pk.h[e] = (bf16)v[e];
            *reinterpret_cast<uint2*>(stg + lrow * RS + (((4 * j + q) ^ (lrow & 7)) << 4) + g * 8) = pk.u;
          }
        }
        wait_lds();
#pragma unroll
        for (int k = 0; k < 32 / RST; ++k) {
          const u32x4 val = *reinterpret_cast<const u32x4*>(stg + (((k * RST) & 7) ? rd1 : rd0) + k * RST * RS);
          // rows past M fall outside the buffer's range; columns past N were sent out of range
          // non-temporal: the output is not re-read by this kernel, and
          // keeping it out of the L2's working set leaves the operand
          // panels there (+2.5% kernel rate on CLIP's QKV / FC1)
          __builtin_amdgcn_raw_buffer_store_b128(val, out_rsrc, st0 + (unsigned)((i * 32 + k * RST) * a.ldo * 2), 0,
                                                 kStoreNT);
        }
        wait_lds();   // the reads are done before the next block row overwrites the staging
      }
      if (has_next) {
        __builtin_amdgcn_s_barrier();   // every wave has read its staging: k-tile 1 may fill the stage
        issue(1, (sb + KT + 1) & 1);
      }
    } else {
    uint2 bq[C::FN];   // the lane's 4 bias values of each block column
#pragma unroll
    for (int j = 0; j < C::FN; ++j) bq[j] = *reinterpret_cast<const uint2*>(slab_b + (j * 32 + pc) * 2);
    wait_lds();
#pragma unroll
    for (int i = 0; i < C::FM; ++i) {
#pragma unroll
      for (int j = 0; j < C::FN; ++j) {
        const int b = i * C::FN + j;
        if constexpr (RES) {
          // loads reach min(b + 1, kResAhead) blocks ahead of block b: the
          // look-ahead grows as finished blocks free their accumulators
          const int upto_prev = b == 0 ? 0 : min(NB - 1, b - 1 + min(b, kResAhead));
          const int upto = min(NB - 1, b + min(b + 1, kResAhead));
#pragma unroll
          for (int d = upto_prev + 1; d <= upto; ++d) rload(d, rq[d % RR]);
        }
        // acc element 4q + e sits at row lrow, column 8q + 4g + e of the block
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<float4*>(slab + lrow * 32 + (((2 * q + g) ^ swz) << 2)) =
              make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
        wait_lds();
        const int n = n0 + wn * C::WN + j * 32 + pc;
        float bv[4];
        {
          union { uint2 u; bf16 h[4]; } bb;
          bb.u = bq[j];
#pragma unroll
          for (int e = 0; e < 4; ++e) bv[e] = (float)bb.h[e] * bias_on;
        }
        // rows past M fall outside the buffer's range; columns past N are sent out of range
        const unsigned st0 = n < a.N ? (unsigned)(((wm * C::WM + i * 32 + prow) * a.ldo + n) * 4) : 0x80000000u;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int r = p * 8 + prow;   // row within the block
          const float4 s0 = *reinterpret_cast<const float4*>(slab + r * 32 + (((pc >> 2) ^ C::sw(r)) << 2));
          float v[4] = {s0.x, s0.y, s0.z, s0.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += bv[e];
          if (act == ACT_GELU) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = gelu_erf(v[e]);
          } else if (act == ACT_QUICKGELU) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = quick_gelu(v[e]);
          }
          if constexpr (RES) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] += __uint_as_float(rq[b % RR][p][e]);
          }
          __builtin_amdgcn_raw_buffer_store_b128(
              (u32x4){__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])},
              out_rsrc, st0 + (unsigned)(p * 8 * a.ldo * 4), 0, 0);
        }
      }
    }
    }
    if constexpr (RES) {
      if (has_next) issue(1, (sb + KT + 1) & 1);   // after the epilogue's loads (see above)
    }
    if (!has_next) break;
    wait_lds();   // the slab reads are done before the next bias DMA rewrites it
    first = false;
    sb = (sb + KT) & 1;
    t = tn;
    m0 = m0n;
    n0 = n0n;
  }
}

template <int BM, int BN, int WGM, int WGN, int ST = 2>
hipError_t launch_tile(const GemmArgs& a, hipStream_t s) {
  using C = Cfg<BM, BN, WGM, WGN, ST>;
  static bool attr = false;   // raise the dynamic-LDS limit once per instantiation
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute((const void*)gemm_bf16_tile_kernel<BM, BN, WGM, WGN, ST>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const long tiles = (long)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_bf16_tile_kernel<BM, BN, WGM, WGN, ST>), dim3((unsigned)tiles), dim3(C::NT), C::LDS, s, a);
  return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN, int OUTF32, int RES = 0, int ROPE = 0>
hipError_t launch_async_t(const GemmArgs& a, hipStream_t s) {
  using C = ACfg<BM, BN, WGM, WGN, OUTF32>;
  auto kern = gemm_bf16_async_kernel<BM, BN, WGM, WGN, OUTF32, RES, ROPE>;
  static int slots = 0;   // co-resident workgroups on this device, found once per instantiation
  if (!slots) {
    hipError_t e = hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess) return e;
    int dev = 0, cus = 0, per_cu = 0;
    if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess) return e;
    if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, (const void*)kern, C::NT, C::LDS)) != hipSuccess)
      return e;
    if (per_cu < 1) return hipErrorInvalidConfiguration;
    slots = cus * per_cu;
  }
  const long tiles = (long)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  if (tiles == 0) return hipSuccess;
  const int grid = (int)(tiles < slots ? tiles : slots);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(C::NT), C::LDS, s, a, (int)tiles);
  return hipGetLastError();
}

template <int BM, int BN, int WGM, int WGN>
hipError_t launch_async(const GemmArgs& a, hipStream_t s) {
  if (a.rope_pos) return launch_async_t<BM, BN, WGM, WGN, 0, 0, 1>(a, s);
  return a.out_f32 ? launch_async_t<BM, BN, WGM, WGN, 1>(a, s) : launch_async_t<BM, BN, WGM, WGN, 0>(a, s);
}

bool al16(const void* p) { return (uintptr_t)p % 16 == 0; }

// The DMA tile kernel's requirements: 16-byte aligned operand rows, K a
// multiple of its k-step, 32-bit byte offsets, and 8-column epilogue chunks
// with 16-byte aligned rows in every epilogue stream.
bool tile_ok(const GemmArgs& a) {
  if (a.stats || a.K % BK || a.N % 8 || a.lda % 8 || a.ldb % 8 || !al16(a.A) || !al16(a.B)) return false;
  if ((double)a.M * a.lda * 2 >= 4294967296.0 || (double)a.N * a.ldb * 2 >= 4294967296.0) return false;
  if (a.out_f32 ? (a.ldo % 4 != 0) : (a.ldo % 8 != 0)) return false;
  if (!al16(a.out) || (a.resid && (a.ldr % 4 || !al16(a.resid)))) return false;
  if (a.pos && (!al16(a.pos) || (a.pos_f32 ? a.ld_pos % 4 : a.ld_pos % 8))) return false;
  return true;
}

// The persistent kernel's buffer resources span one 256-row tile of the output
// (and of the residual) with 32-bit sizes and offsets.
bool tile_rows_fit(const GemmArgs& a) {
  const double lim = 2147483648.0;
  return 256.0 * a.ldo * (a.out_f32 ? 4 : 2) < lim && (!a.resid || 256.0 * a.ldr * 4 < lim);
}

// The persistent asynchronous-epilogue kernel: bias / activation epilogues, two
// to 32 k-tiles.  Past that the epilogue is a small share of a tile and the
// per-tile kernel measured slightly faster (both give the same bits).
bool async_ok(const GemmArgs& a) {
  return tile_ok(a) && tile_rows_fit(a) && !a.resid && !a.pos && a.K >= 2 * BK && a.K <= 32 * BK;
}

// Its residual form (fp32 residual stream, fp32 output: O-projection and FC2), any
// K: the residual read and write are a large share of such a tile, and the
// stores drain under the next tile's k-loop.
bool async_res_ok(const GemmArgs& a) {
  return tile_ok(a) && tile_rows_fit(a) && a.resid && a.out_f32 && !a.pos && a.K >= 2 * BK;
}

}  // namespace

namespace {

// Tile options, fitted to measured launch times on the encoder's shapes.
// `slots` workgroups fit on the chip at once (two 128 x 128 workgroups share
// a CU); a round of them costs area * slots / 256 / eff in units where a
// full round of 256 x 256 tiles costs 65536.  A 128 x 128 launch of at most
// 256 tiles runs one workgroup per CU, at about 0.7 of a shared round.
// The residual forms (fp32 residual read and written, 8 waves at 256 x 256) lose
// more on the smaller tiles: against 256 x 256 the 128 x 128 residual kernel
// measured 0.77-0.81 and the 256 x 128 one 0.69 (video clips' O-projection
// and FC2, M = 32768, N = 1280, timed back to back at each tile size).
struct TileOpt { int bm, bn, slots; double eff; };
constexpr TileOpt kTiles[3] = {{256, 256, 256, 1.00}, {256, 128, 256, 0.80}, {128, 128, 512, 0.90}};
constexpr TileOpt kTilesRes[3] = {{256, 256, 256, 1.00}, {256, 128, 256, 0.69}, {128, 128, 512, 0.78}};

double tile_time(const TileOpt& o, long M, long N) {
  const long tiles = ((M + o.bm - 1) / o.bm) * ((N + o.bn - 1) / o.bn);
  const double round = (double)o.bm * o.bn * (o.slots / 256) / o.eff;
  if (o.slots > 256 && tiles <= 256) return 0.7 * round;
  return (double)((tiles + o.slots - 1) / o.slots) * round;
}

int best_tile(long M, long N, double* t, bool res) {
  const TileOpt* opts = res ? kTilesRes : kTiles;
  int best = 0;
  double best_t = 1e300;
  for (int i = 0; i < 3; ++i) {
    const double ti = tile_time(opts[i], M, N);
    if (ti < best_t) { best_t = ti; best = i; }
  }
  if (t) *t = best_t;
  return best;
}

}  // namespace

// Compute units of the current device (queried once).
int device_cus() {
  static int cus = 0;
  if (!cus) {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) == hipSuccess && hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
      cus = n;
    else
      return 256;
  }
  return cus;
}

bool gemm_bf16_rope_ok(const GemmArgs& a) {
  return tile_ok(a) && !a.out_f32 && !a.resid && !a.pos && a.rope_hd > 0 && a.rope_hd % 8 == 0 && a.rope_hd <= 128 &&
         a.rope_hd_inv == rope_hd_inv(a.rope_hd) && a.rope_cols % a.rope_hd == 0 && a.rope_cols <= a.N && a.N < 65536;
}

hipError_t launch_gemm_bf16(const GemmArgs& a, hipStream_t s, const char** kname) {
  if (a.rope_pos && !gemm_bf16_rope_ok(a)) return hipErrorInvalidValue;
  if (!tile_ok(a)) return launch_gemm_bf16_staged(a, s, kname);
  // Pick the tile by estimated time.  All tiles sum k in the same order, so
  // the choice never changes a result.
  // Launches that leave CUs idle even with 128 x 128 tiles are latency-bound:
  // smaller tiles multiply the workgroups and three stages keep two k-tiles in
  // flight -- 64 x 128 (4 waves of 32 x 64), or 64 x 64 (4 waves of 32 x 32)
  // while 64 x 128 tiles would leave a quarter of the CUs idle.
  // The residual rows a micro-batch half leaves after whole rounds of 256 x 256
  // tiles stay on the persistent residual kernel even when they are few: that
  // launch runs beside the other half's kernels, and measured 1% faster there
  // end to end than the latency tiles (CLIP x64).  Alone on the chip (CLIP x4)
  // the latency tiles are faster.
  const int cus = device_cus();
  const long t128 = (long)((a.M + 127) / 128) * ((a.N + 127) / 128);
  if (t128 <= cus && !(a.beside && a.resid && async_res_ok(a))) {
    // When every tile gets a CU of its own, deeper pipelines (6 stages of 64 x 64,
    // 96 KB; 4 of 64 x 128, 96 KB) keep more k-tiles in flight: one CLIP image
    // +4%, one Whisper clip +1%.  With more tiles than CUs the three-stage forms
    // stay, as two of their workgroups fit in one CU's LDS (6 stages there: two
    // images -17%).
    if ((long)((a.M + 63) / 64) * ((a.N + 127) / 128) * 4 <= 3L * cus) {
      *kname = "gemm_bf16_64x64";
      if ((long)((a.M + 63) / 64) * ((a.N + 63) / 64) <= cus) return launch_tile<64, 64, 2, 2, 6>(a, s);
      return launch_tile<64, 64, 2, 2, 3>(a, s);
    }
    *kname = "gemm_bf16_64x128";
    if ((long)((a.M + 63) / 64) * ((a.N + 127) / 128) <= cus) return launch_tile<64, 128, 2, 2, 4>(a, s);
    return launch_tile<64, 128, 2, 2, 3>(a, s);
  }
  const bool res = a.resid != nullptr;
  if (async_res_ok(a)) switch (best_tile(a.M, a.N, nullptr, true)) {
      case 0:
        *kname = "gemm_bf16_async_res_256x256";   // 8 waves of 64 x 128: 4 KB fp32 slabs
        return launch_async_t<256, 256, 4, 2, 1, 1>(a, s);
      case 1: *kname = "gemm_bf16_async_res_256x128"; return launch_async_t<256, 128, 4, 2, 1, 1>(a, s);
      default: *kname = "gemm_bf16_async_res_128x128"; return launch_async_t<128, 128, 2, 2, 1, 1>(a, s);
    }
  if (async_ok(a)) switch (best_tile(a.M, a.N, nullptr, false)) {
      case 0:   // 16 waves of 64 x 64 with bf16 output (2 KB slabs); the fp32 slabs need 8 waves.
        // The rotary epilogue takes 8 waves of 64 x 128: in 16 waves it spills 19 VGPRs
        // around the tile loop, and 8 measured 2-3.6% faster (video and image QKV)
        *kname = "gemm_bf16_async_256x256";
        if (a.rope_pos) return launch_async_t<256, 256, 4, 2, 0, 0, 1>(a, s);
        return a.out_f32 ? launch_async_t<256, 256, 4, 2, 1>(a, s) : launch_async_t<256, 256, 4, 4, 0>(a, s);
      case 1: *kname = "gemm_bf16_async_256x128"; return launch_async<256, 128, 4, 2>(a, s);
      default: *kname = "gemm_bf16_async_128x128"; return launch_async<128, 128, 2, 2>(a, s);
    }
  switch (best_tile(a.M, a.N, nullptr, res)) {
    case 0: *kname = "gemm_bf16_256x256"; return launch_tile<256, 256, 4, 4>(a, s);
    case 1: *kname = "gemm_bf16_256x128"; return launch_tile<256, 128, 4, 2>(a, s);
    default: *kname = "gemm_bf16_128x128"; return launch_tile<128, 128, 2, 2>(a, s);
  }
}

int gemm_bf16_head_rows(const GemmArgs& a) {
  if (!tile_ok(a)) return 0;
  const long nt = (a.N + 255) / 256, tiles = (long)((a.M + 255) / 256) * nt;
  const long rounds = tiles / 256;
  if (rounds == 0 || tiles % 256 == 0) return 0;
  const long head = rounds * 256 / nt * 256;   // rows covered by whole rounds of 256 x 256 tiles
  if (head <= 0 || head >= a.M) return 0;
  if (a.pos && !a.pos_idx && head % a.pos_period) return 0;
  const bool res = a.resid != nullptr;
  double whole, tail;
  best_tile(a.M, a.N, &whole, res);
  best_tile(a.M - head, a.N, &tail, res);
  const double split = tile_time(kTiles[0], head, a.N) + tail;
  return split < 0.97 * whole ? (int)head : 0;
}

GemmArgs gemm_rows(const GemmArgs& a, int m0, int m1) {
  GemmArgs r = a;
  r.M = m1 - m0;
  r.A = static_cast<const char*>(a.A) + (size_t)m0 * a.lda * 2;
  r.out = static_cast<char*>(a.out) + (size_t)m0 * a.ldo * (a.out_f32 ? 4 : 2);
  if (a.resid) r.resid = a.resid + (size_t)m0 * a.ldr;
  if (a.pos_idx) r.pos_idx = a.pos_idx + m0;
  if (a.rope_pos) r.rope_pos = a.rope_pos + m0;
  return r;
}

}  // namespace eas

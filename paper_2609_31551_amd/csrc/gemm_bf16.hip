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
//  * Two LDS stages of 64 k: tile k+1 streams in while tile k is consumed.
//    The DMA is issued from inline assembly so the compiler does not
//    serialise it against the LDS reads; completion is tracked with explicit
//    s_waitcnt vmcnt and one workgroup barrier per k-step.
//  * v_mfma_f32_32x32x16_bf16, each wave a (BM/WGM) x (BN/WGN) sub-tile of
//    32 x 32 blocks (8 waves of 64 x 128 for the 256 x 256 tile); operand
//    fragments for the next 16-wide k slice are read while the current
//    slice's MFMAs run, and the barrier sits before the last slice so its
//    wait overlaps queued MFMAs.
//  * Tiles are handed out XCD-aware: workgroups are dispatched round-robin
//    over the 8 XCDs, so block b is remapped to give every XCD a contiguous
//    run of output tiles that share A row panels in that XCD's L2.
//  * Fused epilogue through LDS: each wave stages 32 rows of its fp32
//    accumulators, then every lane owns 8 consecutive columns of a row and
//    applies bias, GELU / QuickGELU, a position-table row and the fp32
//    residual before one 16-byte (bf16) or 2 x 16-byte (fp32) store.
//  * Every output element accumulates k in the same order (16-wide MFMA
//    slices, ascending) whatever the tile shape or M, so a
//    request's result does not depend on what else is in the micro-batch.
#include "common.h"

namespace eas {
namespace {

constexpr int BK = 64, ST = 2;

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

template <int BM, int BN, int WGM, int WGN>
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
  static_assert(DPS < 64, "vmcnt range");
  // conflict-free chunk swizzle for 128-byte rows: 16 rows per LDS cycle hit 16 distinct 16-byte slots
  __device__ static int sw(int row) { return (row >> 1) & 7; }
};

// XCD-aware block -> tile index (bijective on [0, nb)).
__device__ __forceinline__ int xcd_tile(int b, int nb) {
  const int per = (nb + 7) / 8, x = b % 8, s = b / 8;
  const int full = nb % 8 == 0 ? 8 : nb % 8;   // XCDs that receive `per` blocks
  return (x < full ? x * per : full * per + (x - full) * (per - 1)) + s;
}

template <int BM, int BN, int WGM, int WGN>
__global__ __launch_bounds__(64 * WGM * WGN) void gemm_bf16_tile_kernel(GemmArgs a) {
  using C = Cfg<BM, BN, WGM, WGN>;
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const unsigned lds0 = (unsigned)(size_t)((__attribute__((address_space(3))) char*)smem);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int tiles_n = (a.N + BN - 1) / BN;
  const int bid = xcd_tile(blockIdx.x, gridDim.x);
  const int m0 = (bid / tiles_n) * BM, n0 = (bid % tiles_n) * BN;
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
      const int gn = min(n0 + r, a.N - 1);
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

  // prologue: tiles 0 .. ST-1 in flight; wait for tile 0
#pragma unroll
  for (int s = 0; s < ST; ++s)
    if (s < KT) issue(s, s);
  if (KT > 1) wait_vm<C::DPS>();   // ST == 2: tile 1 may still be in flight
  else wait_vm<0>();
  __syncthreads();
  load_frags(0, cofs[0], fa[0], fb[0]);

  for (int kt = 0; kt < KT; ++kt) {
    const int st = kt % ST;
#pragma unroll
    for (int h = 0; h < NH - 1; ++h) {
      load_frags(st, cofs[h + 1], fa[(h + 1) & 1], fb[(h + 1) & 1]);
      mma(fa[h & 1], fb[h & 1]);
    }
    if (kt + 1 < KT) {
      // this wave's reads of stage st are done once lgkmcnt drains; tile kt+1
      // (the newest DMA) has landed at vmcnt 0; after the barrier every wave
      // is past stage st, which is refilled with tile kt+ST
      wait_lds();
      wait_vm<0>();
      __builtin_amdgcn_s_barrier();
      if (kt + ST < KT) issue(kt + ST, st);
      load_frags((kt + 1) % ST, cofs[0], fa[NH & 1], fb[NH & 1]);
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

template <int BM, int BN, int WGM, int WGN>
hipError_t launch_tile(const GemmArgs& a, hipStream_t s) {
  using C = Cfg<BM, BN, WGM, WGN>;
  static bool attr = false;   // raise the dynamic-LDS limit once per instantiation
  if (!attr) {
    const hipError_t e = hipFuncSetAttribute((const void*)gemm_bf16_tile_kernel<BM, BN, WGM, WGN>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, C::LDS);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const long tiles = (long)((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((gemm_bf16_tile_kernel<BM, BN, WGM, WGN>), dim3((unsigned)tiles), dim3(C::NT), C::LDS, s, a);
  return hipGetLastError();
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

}  // namespace

hipError_t launch_gemm_bf16(const GemmArgs& a, hipStream_t s, const char** kname) {
  if (!tile_ok(a)) return launch_gemm_bf16_staged(a, s, kname);
  // Pick the tile by estimated time: full-chip rounds (256 CUs; one 256-wide
  // or two 128 x 128 workgroups per CU) times the tile's work over its
  // measured relative efficiency.  All tiles sum k in the same order, so the
  // choice never changes a result.
  struct Opt { int bm, bn, per_cu; double eff; };
  const Opt opts[3] = {{256, 256, 1, 1.00}, {256, 128, 1, 0.80}, {128, 128, 2, 0.65}};
  int best = 0;
  double best_t = 1e300;
  for (int i = 0; i < 3; ++i) {
    const long tiles = (long)((a.M + opts[i].bm - 1) / opts[i].bm) * ((a.N + opts[i].bn - 1) / opts[i].bn);
    const long slots = 256L * opts[i].per_cu;
    const double t = (double)((tiles + slots - 1) / slots) * opts[i].bm * opts[i].bn * opts[i].per_cu / opts[i].eff;
    if (t < best_t) { best_t = t; best = i; }
  }
  switch (best) {
    case 0: *kname = "gemm_bf16_256x256"; return launch_tile<256, 256, 4, 2>(a, s);
    case 1: *kname = "gemm_bf16_256x128"; return launch_tile<256, 128, 4, 2>(a, s);
    default: *kname = "gemm_bf16_128x128"; return launch_tile<128, 128, 2, 2>(a, s);
  }
}

}  // namespace eas

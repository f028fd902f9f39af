// fp32 GEMM for the fp32 mode of the encoder (small models and the fp32
// parity mode).  Same contract as the bf16 MFMA GEMM (GemmArgs): optional
// LayerNorm prologue on an fp32 A, fused bias / activation / position /
// residual epilogue.  Plain FMA on a 64 x 64 tile, k-step 16, each of the 256
// threads owning a 4 x 4 block; k is summed in ascending order for every
// output, so results do not depend on M.
#include "common.h"

namespace eas {
namespace {

constexpr int TM = 64, TN = 64, TK = 16;

__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];
  const int tid = threadIdx.x;
  const int tiles_n = (a.N + TN - 1) / TN;
  const int m0 = (blockIdx.x / tiles_n) * TM, n0 = (blockIdx.x % tiles_n) * TN;
  const int ty = tid / 16, tx = tid % 16;
  const float* A = static_cast<const float*>(a.A);
  const float* B = static_cast<const float*>(a.B);
  const float* g = static_cast<const float*>(a.ln_g);
  const float* b = static_cast<const float*>(a.ln_b);

  float acc[4][4] = {};
  for (int k0 = 0; k0 < a.K; k0 += TK) {
    for (int e = tid; e < TM * TK; e += 256) {
      const int r = e / TK, kk = e % TK;
      const int gm = m0 + r, gk = k0 + kk;
      float v = 0.0f;
      if (gm < a.M && gk < a.K) {
        v = A[(long)gm * a.lda + gk];
        if (a.stats) {
          const float2 st = a.stats[(long)gm * a.ln_group + gk / a.ln_dim];
          const int c = gk % a.ln_dim;
          v = (v - st.x) * st.y * g[c] + b[c];
        }
      }
      As[kk][r] = v;
    }
    for (int e = tid; e < TN * TK; e += 256) {
      const int r = e / TK, kk = e % TK;
      const int gn = n0 + r, gk = k0 + kk;
      Bs[kk][r] = (gn < a.N && gk < a.K) ? B[(long)gn * a.ldb + gk] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }

  const float* bias = static_cast<const float*>(a.bias);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= a.M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n >= a.N) continue;
      float v = apply_act(a.act, acc[i][j] + (bias ? bias[n] : 0.0f));
      if (a.pos) {
        const int pr = a.pos_idx ? a.pos_idx[m] : m % a.pos_period;
        const long pi = (long)pr * a.ld_pos + n;
        v += a.pos_f32 ? static_cast<const float*>(a.pos)[pi] : (float)static_cast<const bf16*>(a.pos)[pi];
      }
      if (a.resid) v += a.resid[(long)m * a.ldr + n];
      const long oi = (long)m * a.ldo + n;
      if (a.out_f32) static_cast<float*>(a.out)[oi] = v;
      else static_cast<bf16*>(a.out)[oi] = (bf16)v;
    }
  }
}

}  // namespace

hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s, const char** kname) {
  const long tiles = (long)((a.M + TM - 1) / TM) * ((a.N + TN - 1) / TN);
  *kname = "gemm_f32_64x64";
  hipLaunchKernelGGL(gemm_f32_kernel, dim3((unsigned)tiles), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace eas

// MFMA issue-rate probe (measurement, not part of the Encode path): every CU
// runs back-to-back v_mfma_f32_32x32x16_bf16 on operands held in registers, so
// no memory traffic takes any of the board's power.  On random finite bf16
// operands the rate settles where the power limit puts it; on all-zero
// operands (no bit toggles) it reaches the clock's full MFMA rate.  The gap
// between the two is what the power budget takes from MFMA-bound work.
#include "common.h"
#include "../../include/eas_encoder.h"

namespace eas {
namespace {

constexpr int kProbeFrags = 8;   // operand fragments cycled through (distinct bits per MFMA)

__device__ __forceinline__ unsigned probe_hash(unsigned x) {
  x ^= x >> 16; x *= 0x7feb352du; x ^= x >> 15; x *= 0x846ca68bu; x ^= x >> 16;
  return x;
}

// A finite bf16 with random sign and mantissa and an exponent in [2^-9, 2^6].
__device__ __forceinline__ unsigned short probe_bits(unsigned h) {
  return (unsigned short)((h & 0x8000u) | ((118u + ((h >> 7) & 15u)) << 7) | (h & 0x7fu));
}

__global__ __launch_bounds__(256) void mfma_probe_kernel(float* out, int iters, int zero) {
  const unsigned t = blockIdx.x * 256u + threadIdx.x;
  bf16x8 fa[kProbeFrags], fb[kProbeFrags];
#pragma unroll
  for (int f = 0; f < kProbeFrags; ++f)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const unsigned h = probe_hash(t * 131u + f * 17u + e * 7u + 1u);
      fa[f][e] = __builtin_bit_cast(bf16, (unsigned short)(zero ? 0u : probe_bits(h)));
      fb[f][e] = __builtin_bit_cast(bf16, (unsigned short)(zero ? 0u : probe_bits(probe_hash(h))));
    }
  f32x16 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[j][e] = 0.0f;
  for (int i = 0; i < iters; ++i)
#pragma unroll
    for (int f = 0; f < kProbeFrags; ++f)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[f], fb[(f + j) % kProbeFrags], acc[j], 0, 0, 0);
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[j][e];
  out[t] = s;   // keeps the MFMAs live
}

}  // namespace
}  // namespace eas

extern "C" eas_status eas_mfma_rate_probe(int32_t zero_operands, int32_t iters, double* tflops, void* stream) {
  if (!tflops || iters < 1 || iters > (1 << 20)) return EAS_ERR_INVALID_ARG;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
    return EAS_ERR_HIP;
  const int grid = cus;   // one workgroup of 4 waves (one per SIMD) per CU
  hipStream_t s = static_cast<hipStream_t>(stream);
  float* out = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  eas_status st = EAS_ERR_HIP;
  if (hipMalloc(&out, (size_t)grid * 256 * sizeof(float)) == hipSuccess && hipEventCreate(&e0) == hipSuccess &&
      hipEventCreate(&e1) == hipSuccess) {
    // one warm-up launch brings the clock to its steady state, then one timed
    hipLaunchKernelGGL(eas::mfma_probe_kernel, dim3(grid), dim3(256), 0, s, out, iters, zero_operands != 0);
    float ms = 0.0f;
    if (hipGetLastError() == hipSuccess && hipEventRecord(e0, s) == hipSuccess) {
      hipLaunchKernelGGL(eas::mfma_probe_kernel, dim3(grid), dim3(256), 0, s, out, iters, zero_operands != 0);
      if (hipGetLastError() == hipSuccess && hipEventRecord(e1, s) == hipSuccess &&
          hipEventSynchronize(e1) == hipSuccess && hipEventElapsedTime(&ms, e0, e1) == hipSuccess && ms > 0.0f) {
        const double flops = (double)grid * 4 * iters * eas::kProbeFrags * 4 * 2.0 * 32 * 32 * 16;
        *tflops = flops / (ms * 1e-3) / 1e12;
        st = EAS_OK;
      }
    }
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (out) (void)hipFree(out);
  return st;
}

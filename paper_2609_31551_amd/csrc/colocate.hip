// Compute-unit reservation for the co-location profile (Section 3.4, dynamic
// SM partitioning): encode latency is measured while part of the GPU is held
// by other work.  The paper confines each process to an SM subset with TPC
// masks; here the held share is taken by occupancy instead: each workgroup of
// the reservation kernel claims one whole CU -- the CU's 160 KB of LDS and,
// with four 128-VGPR waves per SIMD, its whole register file -- so no
// workgroup of any other kernel can be placed there until it exits.
#include "common.h"
#include "../../include/eas_colocate.h"

namespace eas {
namespace {

constexpr int kHoldThreads = 1024;          // 16 waves: 4 per SIMD
constexpr int kHoldLds = 160 * 1024;        // all of a CU's LDS

// Thread 0 marks its block as resident in started[block] (host memory), then
// sleeps until *release != 0 or `budget` ticks of the constant-rate wall
// clock have passed; the other waves wait at the barrier.  Every wave exits
// by the budget at the latest.  The flag is read over PCIe about every 60 us
// (16 of the longest sleeps between reads): polled every few microseconds by
// two hundred blocks, those reads slowed the other kernels' dispatch.
__global__ __launch_bounds__(kHoldThreads) void hold_cu_kernel(int* started, const int* release, long long budget) {
  asm volatile("" ::: "v127");   // the register allocation covers v0..v127: four waves fill a SIMD
  if (threadIdx.x == 0) {
    __hip_atomic_store(started + blockIdx.x, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    const long long t0 = wall_clock64();
    while (wall_clock64() - t0 < budget &&
           __hip_atomic_load(release, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM) == 0)
      for (int i = 0; i < 16; ++i) __builtin_amdgcn_s_sleep(127);
  }
  __syncthreads();
}

}  // namespace
}  // namespace eas

// gfx950 groups its compute units into shader engines of 8 (32 on a 256-CU
// MI355X); a share that leaves some shader engine without a free CU stalls
// every other kernel behind it, so the reservation keeps one per engine free.
constexpr int kCusPerShaderEngine = 8;

extern "C" int32_t eas_cu_reserve_max(int32_t device_cus) {
  return device_cus <= 0 ? 0 : device_cus - (device_cus + kCusPerShaderEngine - 1) / kCusPerShaderEngine;
}

extern "C" eas_status eas_cu_reserve(int32_t n_cus, double max_seconds, int32_t* started, const int32_t* release,
                                     void* stream) {
  if (!started || !release || !(max_seconds > 0.0) || max_seconds > 60.0) return EAS_ERR_INVALID_ARG;
  int dev = 0, cus = 0, khz = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess || khz <= 0)
    return EAS_ERR_HIP;
  if (n_cus < 1 || n_cus > eas_cu_reserve_max(cus)) return EAS_ERR_INVALID_ARG;
  static bool attr = false;
  if (!attr) {
    if (hipFuncSetAttribute((const void*)eas::hold_cu_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            eas::kHoldLds) != hipSuccess)
      return EAS_ERR_HIP;
    attr = true;
  }
  const long long budget = (long long)(max_seconds * 1000.0 * khz);
  hipLaunchKernelGGL(eas::hold_cu_kernel, dim3(n_cus), dim3(eas::kHoldThreads), eas::kHoldLds,
                     static_cast<hipStream_t>(stream), (int*)started, (const int*)release, budget);
  return hipGetLastError() == hipSuccess ? EAS_OK : EAS_ERR_HIP;
}

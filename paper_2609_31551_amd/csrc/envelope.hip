// Per-destination embedding envelopes (paper Section 3.3): a device gather
// from the encoder's request-ordered output into destination-grouped blocks.
// One launch copies every request of the micro-batch in 16-byte chunks; each
// workgroup moves a run of 1024 chunks of one request (the request's row
// offsets travel by value in the kernel arguments).
#include "common.h"
#include "../../include/eas_router.h"

namespace eas {
namespace {

constexpr int kChunksPerThread = 4, kThreads = 256, kChunksPerBlock = kChunksPerThread * kThreads;

struct GatherArgs {
  int n;
  long src_chunk[kMaxSeqs + 1];   // prefix sums of each request's 16-byte chunks (source order)
  long dst_chunk[kMaxSeqs];       // first destination chunk of each request
  int block0[kMaxSeqs + 1];       // prefix sums of each request's workgroups
};

// Workgroup b copies up to kChunksPerBlock consecutive chunks of one request;
// the request is found once per workgroup.
__global__ __launch_bounds__(kThreads) void envelope_gather_kernel(const uint4* src, uint4* dst, GatherArgs a) {
  const int b = blockIdx.x;
  int lo = 0, hi = a.n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.block0[mid] <= b) lo = mid; else hi = mid - 1;
  }
  const long first = a.src_chunk[lo] + (long)(b - a.block0[lo]) * kChunksPerBlock;
  const long end = a.src_chunk[lo + 1];
  const long shift = a.dst_chunk[lo] - a.src_chunk[lo];
  uint4 v[kChunksPerThread];
#pragma unroll
  for (int j = 0; j < kChunksPerThread; ++j) {
    const long c = first + j * kThreads + threadIdx.x;
    if (c < end) v[j] = src[c];
  }
#pragma unroll
  for (int j = 0; j < kChunksPerThread; ++j) {
    const long c = first + j * kThreads + threadIdx.x;
    if (c < end) dst[c + shift] = v[j];
  }
}

}  // namespace
}  // namespace eas

extern "C" eas_status eas_envelope_gather(const void* src, const int64_t* src_rows, const int64_t* req_rows,
                                          int32_t n_req, int64_t row_bytes, void* dst, void* stream) {
  using namespace eas;
  if (n_req < 0 || n_req > kMaxSeqs || row_bytes <= 0 || row_bytes % 16 || (n_req > 0 && (!src_rows || !req_rows)))
    return EAS_ERR_INVALID_ARG;
  if (n_req == 0) return EAS_OK;
  if (!src || !dst || (uintptr_t)src % 16 || (uintptr_t)dst % 16) return EAS_ERR_INVALID_ARG;
  if (src_rows[0] != 0) return EAS_ERR_INVALID_ARG;
  GatherArgs a;
  a.n = n_req;
  const long cpr = row_bytes / 16;   // chunks per row
  a.src_chunk[0] = 0;
  a.block0[0] = 0;
  for (int i = 0; i < n_req; ++i) {
    const int64_t r = src_rows[i + 1] - src_rows[i];
    if (r < 0 || req_rows[i] < 0) return EAS_ERR_INVALID_ARG;
    a.src_chunk[i + 1] = a.src_chunk[i] + r * cpr;
    a.dst_chunk[i] = req_rows[i] * cpr;
    const long blocks = (r * cpr + kChunksPerBlock - 1) / kChunksPerBlock;
    if (a.block0[i] + blocks > 0x7fffffffL) return EAS_ERR_CAPACITY;
    a.block0[i + 1] = a.block0[i] + (int)blocks;
  }
  if (a.block0[n_req] == 0) return EAS_OK;
  hipLaunchKernelGGL(envelope_gather_kernel, dim3((unsigned)a.block0[n_req]), dim3(kThreads), 0, (hipStream_t)stream,
                     (const uint4*)src, (uint4*)dst, a);
  return hipGetLastError() == hipSuccess ? EAS_OK : EAS_ERR_HIP;
}

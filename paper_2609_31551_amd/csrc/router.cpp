// Deficit-counter router and envelope plan (paper Section 3.3).  Host-only;
// the C ABI is declared in include/eas_router.h.
#include "../../include/eas_router.h"

#include <cmath>
#include <new>
#include <vector>

namespace {
// 1.0 in the accumulator's fixed point: multiples of 1 / (2^20 10^9) hold
// every decimal ratio of up to 9 digits and every 20-bit binary ratio exactly
constexpr uint64_t kOne = (1ull << 20) * 1000000000ull;
}

struct eas_router {
  uint64_t s = 0;       // offload ratio, in units of 1 / kOne
  uint64_t d = 0;       // accumulator, same units; below kOne between requests
  int64_t routed = 0, remote = 0;
};

extern "C" {

eas_status eas_router_create(double offload_ratio, eas_router** out) {
  if (!out) return EAS_ERR_INVALID_ARG;
  *out = nullptr;
  if (!(offload_ratio >= 0.0 && offload_ratio <= 1.0)) return EAS_ERR_INVALID_ARG;
  eas_router* r = new (std::nothrow) eas_router();
  if (!r) return EAS_ERR_CAPACITY;
  r->s = (uint64_t)std::llround(offload_ratio * (double)kOne);
  *out = r;
  return EAS_OK;
}

void eas_router_destroy(eas_router* r) { delete r; }

eas_status eas_router_ratio(const eas_router* r, double* s) {
  if (!r || !s) return EAS_ERR_INVALID_ARG;
  *s = (double)r->s / (double)kOne;
  return EAS_OK;
}

eas_status eas_router_route(eas_router* r, int64_t n, uint8_t* remote) {
  if (!r || n < 0 || (n > 0 && !remote)) return EAS_ERR_INVALID_ARG;
  for (int64_t i = 0; i < n; ++i) {
    r->d += r->s;
    const bool far = r->d >= kOne;
    if (far) r->d -= kOne;
    remote[i] = far;
    r->remote += far;
  }
  r->routed += n;
  return EAS_OK;
}

eas_status eas_router_counts(const eas_router* r, int64_t* routed, int64_t* remote) {
  if (!r || !routed || !remote) return EAS_ERR_INVALID_ARG;
  *routed = r->routed;
  *remote = r->remote;
  return EAS_OK;
}

eas_status eas_envelope_plan(int32_t n_req, const int32_t* dest, int32_t n_dest, const int64_t* rows,
                             int32_t* order, int64_t* dest_rows, int64_t* req_rows) {
  if (n_req < 0 || n_dest < 1 || (n_req > 0 && (!dest || !rows || !order || !req_rows)) || !dest_rows)
    return EAS_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n_req; ++i)
    if (dest[i] < 0 || dest[i] >= n_dest || rows[i] < 0) return EAS_ERR_INVALID_ARG;
  std::vector<int64_t> total(n_dest, 0);
  for (int32_t i = 0; i < n_req; ++i) total[dest[i]] += rows[i];
  dest_rows[0] = 0;
  for (int32_t d = 0; d < n_dest; ++d) dest_rows[d + 1] = dest_rows[d] + total[d];
  std::vector<int64_t> next(dest_rows, dest_rows + n_dest);   // running row cursor per destination
  std::vector<int32_t> slot(n_dest, 0);                        // running request count per destination
  std::vector<int32_t> first(n_dest + 1, 0);
  for (int32_t i = 0; i < n_req; ++i) ++first[dest[i] + 1];
  for (int32_t d = 0; d < n_dest; ++d) first[d + 1] += first[d];
  for (int32_t i = 0; i < n_req; ++i) {
    const int32_t d = dest[i];
    req_rows[i] = next[d];
    next[d] += rows[i];
    order[first[d] + slot[d]++] = i;
  }
  return EAS_OK;
}

}  // extern "C"

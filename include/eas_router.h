/*
 * eas_router.h -- C ABI of the deficit-counter router and of the
 * per-destination embedding envelopes (libeas.so).
 *
 * Router (paper Section 3.3, "Deficit-controlled routing").  A fraction s of
 * the requests leaving the encode worker has its prefill sent to a remote
 * prefill worker, the rest to the co-resident local one.  One accumulator d,
 * initially 0: for each request d += s; if d >= 1 the request goes remote and
 * d -= 1, otherwise it stays local.  After n requests the remote count is
 * floor(n s) (within 1 of n s), and no more than ceil(1/(1-s)) consecutive
 * remote or ceil(1/s) consecutive local decisions occur.  Here d is held in
 * fixed point, in units of 1 / (2^20 * 10^9), so those identities hold exactly
 * for every n: s is rounded to the nearest such multiple, which is exact for
 * decimal ratios of up to 9 digits (eas_router_ratio reports the value used).
 *
 * Envelopes (Section 3.3, "Envelope-based embedding transfer").  All
 * embeddings of a micro-batch bound for the same destination travel as one
 * contiguous block.  eas_envelope_plan gives the stable order that groups
 * requests by destination and the row offsets of every block; encoding the
 * micro-batch in that order makes the encoder's output the grouped envelopes
 * directly (a request's rows do not depend on its place in the batch).
 * eas_envelope_gather builds the envelopes on the device from an output that
 * is in request order.
 *
 * Conventions as in eas_encoder.h: every call returns an eas_status, argument
 * errors are found before anything happens, host arrays are caller-owned.
 */
#ifndef EAS_ROUTER_H
#define EAS_ROUTER_H

#include <stdint.h>

#include "eas_encoder.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct eas_router eas_router;

/* offload_ratio s in [0, 1]. */
eas_status eas_router_create(double offload_ratio, eas_router** out);
void eas_router_destroy(eas_router* r);   /* NULL-safe */

/* The ratio actually used (s rounded to a multiple of 1 / (2^20 * 10^9)). */
eas_status eas_router_ratio(const eas_router* r, double* s);

/* Decisions for the next n requests: remote[i] = 1 (remote prefill) or 0
 * (local prefill); remote is a host array of n bytes. */
eas_status eas_router_route(eas_router* r, int64_t n, uint8_t* remote);

/* Requests routed so far and how many of them went remote. */
eas_status eas_router_counts(const eas_router* r, int64_t* routed, int64_t* remote);

/* Envelope plan for a micro-batch of n_req requests (host arrays):
 *   dest[i] in [0, n_dest)       destination of request i,
 *   rows[i] >= 0                 its embedding rows.
 * Outputs:
 *   order[k]                     request placed k-th (grouped by destination,
 *                                request order kept inside a group),
 *   dest_rows[d], d <= n_dest    row offset of destination d's block
 *                                (dest_rows[n_dest] = total rows),
 *   req_rows[i]                  row offset of request i in the grouped layout. */
eas_status eas_envelope_plan(int32_t n_req, const int32_t* dest, int32_t n_dest, const int64_t* rows,
                             int32_t* order, int64_t* dest_rows, int64_t* req_rows);

/* Device copy into the grouped layout: request i's rows src_rows[i] ..
 * src_rows[i+1] of `src` (device, request order, row_bytes per row) go to
 * rows req_rows[i] .. of `dst` (device).  src_rows (n_req + 1 values) and
 * req_rows are host arrays; n_req <= EAS_MAX_SEQS; row_bytes, src and dst
 * 16-byte aligned.  Enqueued on `stream`; src and dst must not overlap. */
eas_status eas_envelope_gather(const void* src, const int64_t* src_rows, const int64_t* req_rows, int32_t n_req,
                               int64_t row_bytes, void* dst, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* EAS_ROUTER_H */

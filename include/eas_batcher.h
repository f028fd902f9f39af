/*
 * eas_batcher.h -- C ABI of the load-adaptive micro-batcher that feeds the
 * Encode-stage encoder (libeas.so).
 *
 * The rule (paper Section 3.2, "Poisson-gap dispatch rule", Eq. 5).  The
 * encode batch bound B is fixed offline; at run time the batcher decides when
 * a partial batch leaves.  With per-worker arrival rate lambda and a target
 * probability p of filling a batch, Poisson arrivals fill a batch when each of
 * the B-1 inter-arrival gaps after its first request is at most g, which
 * happens with probability (1 - exp(-lambda g))^(B-1).  Setting that to p:
 *     kappa = -ln(1 - p^(1/(B-1))),   g = kappa / lambda.
 * A batch is dispatched as soon as any of these holds:
 *     its size reaches B, or
 *     the idle time since its latest arrival exceeds g, or
 *     the age since its first arrival exceeds the hard cap A (1 s in the paper).
 * The paper uses p = 0.6.
 *
 * Time is supplied by the caller (seconds, any fixed origin), so the batcher
 * is deterministic and the same object serves a live loop (pass a monotonic
 * clock) and a trace replay.  A batch dispatched by timeout leaves at
 *     deadline = min(latest_arrival + g, first_arrival + A)
 * (the instant "idle > g" or "age > A" first holds); an arrival at exactly the
 * deadline still joins the batch (the conditions are strict).  B = 1
 * dispatches every arrival on its own.
 *
 * Conventions: host-only, no HIP calls; the handle is not thread-safe (one
 * caller at a time); every call returns an eas_status (eas_encoder.h), and
 * argument errors leave the handle unchanged.
 */
#ifndef EAS_BATCHER_H
#define EAS_BATCHER_H

#include <stdint.h>

#include "eas_encoder.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int batch_bound;        /* B >= 1 (at most EAS_MAX_SEQS when it feeds one encoder call) */
  double fill_prob;       /* p in (0, 1); ignored when B == 1 */
  double arrival_rate;    /* lambda > 0, requests per second for this worker */
  double max_age;         /* A > 0 seconds; the paper's 1.0 */
} eas_batcher_config;

/* kappa of Eq. 5 for B >= 2 and 0 < p < 1 (written to *kappa). */
eas_status eas_poisson_gap_kappa(int batch_bound, double fill_prob, double* kappa);

/* g = kappa / lambda (seconds); +infinity is never returned: B == 1 gives 0. */
eas_status eas_poisson_gap_threshold(int batch_bound, double fill_prob, double arrival_rate, double* gap);

typedef struct eas_batcher eas_batcher;

/* Validates the config and allocates the handle (host memory only). */
eas_status eas_batcher_create(const eas_batcher_config* cfg, eas_batcher** out);
void eas_batcher_destroy(eas_batcher* b);   /* NULL-safe */

/* Re-derives g for a new arrival-rate estimate (the batch in progress keeps
 * its requests; its deadline moves with g). */
eas_status eas_batcher_set_rate(eas_batcher* b, double arrival_rate);

/* The gap threshold g in seconds. */
eas_status eas_batcher_gap(const eas_batcher* b, double* gap);

/* Request `id` arrives at time t (t must not precede the previous arrival).
 * Any pending timeout dispatch due at or before t must have been collected
 * first (eas_batcher_poll); otherwise EAS_ERR_INVALID_ARG.  *dispatch = 1
 * when the batch is now full and must leave at t. */
eas_status eas_batcher_arrive(eas_batcher* b, double t, int64_t id, int* dispatch);

/* *deadline = when the open batch leaves if nothing else arrives;
 * +infinity when no batch is open. */
eas_status eas_batcher_deadline(const eas_batcher* b, double* deadline);

/* *dispatch = 1 when, at time t, the open batch must leave (t > deadline, or
 * t == deadline: the strict conditions hold just after it). */
eas_status eas_batcher_poll(const eas_batcher* b, double t, int* dispatch);

/* Removes the open batch: its ids in arrival order go to ids[0 .. *n) (host,
 * capacity `cap` >= its size, else EAS_ERR_CAPACITY and nothing removed),
 * *first_arrival gets its first arrival time (may be NULL). */
eas_status eas_batcher_take(eas_batcher* b, int64_t* ids, int cap, int* n, double* first_arrival);

/* Number of requests in the open batch. */
eas_status eas_batcher_size(const eas_batcher* b, int* n);

/* Trace replay against one encode worker.  `arrivals` (host, n_req values,
 * non-decreasing seconds) are fed through the rule of `cfg`; each dispatched
 * batch of size s joins a FIFO in front of a single encode server that is
 * busy service_s[s] seconds per batch (service_s: host, batch_bound + 1
 * values, entry 0 unused).  Outputs (host, caller-owned):
 *   dispatch_t[i], done_t[i]  -- request i's batch dispatch and completion time,
 *   batch_size[i]              -- size of request i's batch,
 *   *n_batches                 -- number of batches.
 * Any output pointer may be NULL. */
eas_status eas_batcher_simulate(const eas_batcher_config* cfg, const double* arrivals, int64_t n_req,
                                const double* service_s, double* dispatch_t, double* done_t,
                                int32_t* batch_size, int64_t* n_batches);

#ifdef __cplusplus
}
#endif

#endif /* EAS_BATCHER_H */

// Load-adaptive micro-batcher (paper Section 3.2, Eq. 5) and its trace
// replay against one encode worker.  Host-only; the C ABI is declared in
// include/eas_batcher.h.
#include "../../include/eas_batcher.h"

#include <cmath>
#include <limits>
#include <new>
#include <vector>

namespace {

constexpr double kInf = std::numeric_limits<double>::infinity();

bool config_ok(const eas_batcher_config* c) {
  if (!c || c->batch_bound < 1) return false;
  if (c->batch_bound > 1 && !(c->fill_prob > 0.0 && c->fill_prob < 1.0)) return false;
  return c->arrival_rate > 0.0 && std::isfinite(c->arrival_rate) && c->max_age > 0.0;
}

// kappa = -ln(1 - p^(1/(B-1))): the gap, in units of the mean inter-arrival
// time, below which all B-1 gaps fall with probability p.
double kappa_of(int B, double p) { return -std::log(1.0 - std::pow(p, 1.0 / (B - 1))); }

double gap_of(const eas_batcher_config& c) {
  return c.batch_bound == 1 ? 0.0 : kappa_of(c.batch_bound, c.fill_prob) / c.arrival_rate;
}

}  // namespace

struct eas_batcher {
  eas_batcher_config cfg;
  double gap = 0.0;
  std::vector<int64_t> ids;   // open batch, arrival order
  double first = 0.0, last = 0.0;
  double prev = -kInf;        // latest arrival seen

  double deadline() const { return ids.empty() ? kInf : std::fmin(last + gap, first + cfg.max_age); }
};

extern "C" {

eas_status eas_poisson_gap_kappa(int batch_bound, double fill_prob, double* kappa) {
  if (!kappa || batch_bound < 2 || !(fill_prob > 0.0 && fill_prob < 1.0)) return EAS_ERR_INVALID_ARG;
  *kappa = kappa_of(batch_bound, fill_prob);
  return EAS_OK;
}

eas_status eas_poisson_gap_threshold(int batch_bound, double fill_prob, double arrival_rate, double* gap) {
  eas_batcher_config c{batch_bound, fill_prob, arrival_rate, 1.0};
  if (!gap || !config_ok(&c)) return EAS_ERR_INVALID_ARG;
  *gap = gap_of(c);
  return EAS_OK;
}

eas_status eas_batcher_create(const eas_batcher_config* cfg, eas_batcher** out) {
  if (!out) return EAS_ERR_INVALID_ARG;
  *out = nullptr;
  if (!config_ok(cfg)) return EAS_ERR_INVALID_ARG;
  eas_batcher* b = new (std::nothrow) eas_batcher();
  if (!b) return EAS_ERR_CAPACITY;
  b->cfg = *cfg;
  b->gap = gap_of(*cfg);
  b->ids.reserve(cfg->batch_bound);
  *out = b;
  return EAS_OK;
}

void eas_batcher_destroy(eas_batcher* b) { delete b; }

eas_status eas_batcher_set_rate(eas_batcher* b, double arrival_rate) {
  if (!b) return EAS_ERR_INVALID_ARG;
  eas_batcher_config c = b->cfg;
  c.arrival_rate = arrival_rate;
  if (!config_ok(&c)) return EAS_ERR_INVALID_ARG;
  b->cfg = c;
  b->gap = gap_of(c);
  return EAS_OK;
}

eas_status eas_batcher_gap(const eas_batcher* b, double* gap) {
  if (!b || !gap) return EAS_ERR_INVALID_ARG;
  *gap = b->gap;
  return EAS_OK;
}

eas_status eas_batcher_arrive(eas_batcher* b, double t, int64_t id, int* dispatch) {
  if (!b || !dispatch || !std::isfinite(t) || t < b->prev) return EAS_ERR_INVALID_ARG;
  if (t > b->deadline()) return EAS_ERR_INVALID_ARG;   // a timeout dispatch was due first
  if (b->ids.empty()) b->first = t;
  b->ids.push_back(id);
  b->last = b->prev = t;
  *dispatch = (int)b->ids.size() >= b->cfg.batch_bound;
  return EAS_OK;
}

eas_status eas_batcher_deadline(const eas_batcher* b, double* deadline) {
  if (!b || !deadline) return EAS_ERR_INVALID_ARG;
  *deadline = b->deadline();
  return EAS_OK;
}

eas_status eas_batcher_poll(const eas_batcher* b, double t, int* dispatch) {
  if (!b || !dispatch) return EAS_ERR_INVALID_ARG;
  *dispatch = !b->ids.empty() && t >= b->deadline();
  return EAS_OK;
}

eas_status eas_batcher_take(eas_batcher* b, int64_t* ids, int cap, int* n, double* first_arrival) {
  if (!b || !n || (cap > 0 && !ids) || cap < 0) return EAS_ERR_INVALID_ARG;
  const int sz = (int)b->ids.size();
  if (sz > cap) return EAS_ERR_CAPACITY;
  for (int i = 0; i < sz; ++i) ids[i] = b->ids[i];
  *n = sz;
  if (first_arrival) *first_arrival = sz ? b->first : kInf;
  b->ids.clear();
  return EAS_OK;
}

eas_status eas_batcher_size(const eas_batcher* b, int* n) {
  if (!b || !n) return EAS_ERR_INVALID_ARG;
  *n = (int)b->ids.size();
  return EAS_OK;
}

eas_status eas_batcher_simulate(const eas_batcher_config* cfg, const double* arrivals, int64_t n_req,
                                const double* service_s, double* dispatch_t, double* done_t,
                                int32_t* batch_size, int64_t* n_batches) {
  if (!config_ok(cfg) || n_req < 0 || (n_req > 0 && !arrivals) || !service_s) return EAS_ERR_INVALID_ARG;
  for (int s = 1; s <= cfg->batch_bound; ++s)
    if (!(service_s[s] >= 0.0) || !std::isfinite(service_s[s])) return EAS_ERR_INVALID_ARG;
  for (int64_t i = 0; i < n_req; ++i)
    if (!std::isfinite(arrivals[i]) || (i && arrivals[i] < arrivals[i - 1])) return EAS_ERR_INVALID_ARG;

  eas_batcher b;
  b.cfg = *cfg;
  b.gap = gap_of(*cfg);
  double server_free = -kInf;
  int64_t batches = 0;
  // one FIFO server: a batch starts when both it and the server are ready
  auto emit = [&](double t) {
    const int s = (int)b.ids.size();
    const double done = std::fmax(t, server_free) + service_s[s];
    server_free = done;
    for (int64_t id : b.ids) {
      if (dispatch_t) dispatch_t[id] = t;
      if (done_t) done_t[id] = done;
      if (batch_size) batch_size[id] = s;
    }
    b.ids.clear();
    ++batches;
  };
  for (int64_t i = 0; i < n_req; ++i) {
    const double t = arrivals[i];
    if (t > b.deadline()) emit(b.deadline());   // the open batch timed out before this arrival
    if (b.ids.empty()) b.first = t;
    b.ids.push_back(i);
    b.last = t;
    if ((int)b.ids.size() >= cfg->batch_bound) emit(t);
  }
  if (!b.ids.empty()) emit(b.deadline());
  if (n_batches) *n_batches = batches;
  return EAS_OK;
}

}  // extern "C"

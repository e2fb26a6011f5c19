// Host side only: block-grained scheduling (Algorithm 1) and compute-aware
// admission (paragraph "Compute-aware admission control", Eq. 1), the loop
// that drives the step kernels between block boundaries. No device code.
//
// Readings where the paper is silent (the same ones the reference follows):
// the pending queue is ascending in prompt length by default (ties in arrival
// order), descending and arrival order are options; a refill alternates two
// moves until neither admits anything: admit every sand-filling candidate
// (row width p + L no wider than the current box) whose admission keeps Eq. 1
// within the budget, scanning the whole queue, then admit the head of the
// queue if it fits (possibly widening the box, which can turn further queued
// requests into sand fills); the Fixed policy admits from the
// head while fewer than the cap are active; an admitted request takes the
// lowest free row of the physical box, right-aligned (off = width - (p + g)).
#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "bs_internal.h"

namespace {

thread_local std::string g_sched_err;

int sfail(int st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_sched_err = buf;
  return st;
}

struct SReq {
  int32_t id, p, g, b;
  int32_t row;
  int64_t seq;
  int32_t K(int L) const { return (g + L - 1) / L; }
  int64_t width(int L) const { return (int64_t)p + (int64_t)(b + 1) * L; }
};

}  // namespace

struct bs_sched {
  bs_sched_config cfg{};
  std::vector<SReq> pending;        // kept in queue order
  std::vector<SReq> active;         // admission order
  std::vector<unsigned char> used;  // rows in use
  int64_t seq = 0;
  int64_t cycles = 0, sum_active = 0, n_finished = 0;
  // plan storage, valid until the next refill
  std::vector<bs_req_desc> descs;
  std::vector<int32_t> ids, admitted;
  std::vector<bs_copy_seg> segs;
};

namespace {

bool queue_before(const bs_sched_config& c, const SReq& x, const SReq& y) {
  if (c.order == BS_ORDER_ASCENDING && x.p != y.p) return x.p < y.p;
  if (c.order == BS_ORDER_DESCENDING && x.p != y.p) return x.p > y.p;
  return x.seq < y.seq;
}

// Eq. 1 of the active set plus an optional candidate entering at block 0.
int64_t eq1_cost(const bs_sched* s, const SReq* cand) {
  const int L = s->cfg.L;
  int64_t n = (int64_t)s->active.size(), w = 0;
  for (const SReq& r : s->active) w = std::max(w, r.width(L));
  if (cand) {
    ++n;
    w = std::max(w, (int64_t)cand->p + L);
  }
  return n * w;
}

int free_row(const bs_sched* s) {
  for (int r = 0; r < s->cfg.rows; ++r)
    if (!s->used[r]) return r;
  return -1;
}

void take(bs_sched* s, size_t i) {
  SReq r = s->pending[i];
  s->pending.erase(s->pending.begin() + (ptrdiff_t)i);
  r.row = free_row(s);
  s->used[r.row] = 1;
  s->active.push_back(r);
  s->admitted.push_back(r.id);
}

}  // namespace

extern "C" {

const char* bs_sched_last_error(void) { return g_sched_err.c_str(); }

int bs_sched_create(bs_sched** out, const bs_sched_config* cfg) {
  if (!out || !cfg) return sfail(BS_ERR_INVALID_ARG, "NULL argument");
  *out = nullptr;
  const bs_sched_config& c = *cfg;
  if (c.L < 1 || c.rows < 1 || c.width < 1) return sfail(BS_ERR_INVALID_ARG, "L, rows and width must be >= 1");
  if (c.policy != BS_SCHED_BUDGET && c.policy != BS_SCHED_FIXED) return sfail(BS_ERR_INVALID_ARG, "bad policy %d", c.policy);
  if (c.policy == BS_SCHED_BUDGET && c.budget < 1) return sfail(BS_ERR_INVALID_ARG, "budget must be >= 1");
  if (c.policy == BS_SCHED_FIXED && c.fixed_batch < 1) return sfail(BS_ERR_INVALID_ARG, "fixed_batch must be >= 1");
  if (c.order != BS_ORDER_ASCENDING && c.order != BS_ORDER_DESCENDING && c.order != BS_ORDER_ARRIVAL)
    return sfail(BS_ERR_INVALID_ARG, "bad queue order %d", c.order);
  bs_sched* s = new bs_sched();
  s->cfg = c;
  s->used.assign((size_t)c.rows, 0);
  *out = s;
  return BS_OK;
}

int bs_sched_destroy(bs_sched* s) {
  delete s;
  return BS_OK;
}

int bs_sched_submit(bs_sched* s, const bs_sched_request* reqs, int n) {
  if (!s) return sfail(BS_ERR_INVALID_ARG, "scheduler is NULL");
  if (n < 0 || (n > 0 && !reqs)) return sfail(BS_ERR_INVALID_ARG, "bad request array");
  const bs_sched_config& c = s->cfg;
  for (int i = 0; i < n; ++i) {
    const bs_sched_request& r = reqs[i];
    if (r.p < 0 || r.g < 1) return sfail(BS_ERR_DESCRIPTOR, "request %d: p=%d g=%d", r.id, r.p, r.g);
    if ((int64_t)r.p + r.g > c.width)
      return sfail(BS_ERR_DESCRIPTOR, "request %d: p + g = %d exceeds the box width %d", r.id, r.p + r.g, c.width);
    if (c.policy == BS_SCHED_BUDGET && (int64_t)r.p + c.L > c.budget)
      return sfail(BS_ERR_DESCRIPTOR, "request %d: p + L = %d exceeds the budget alone", r.id, r.p + c.L);
  }
  for (int i = 0; i < n; ++i) {
    SReq q{reqs[i].id, reqs[i].p, reqs[i].g, 0, -1, s->seq++};
    auto at = std::upper_bound(s->pending.begin(), s->pending.end(), q,
                               [&](const SReq& x, const SReq& y) { return queue_before(c, x, y); });
    s->pending.insert(at, q);
  }
  return BS_OK;
}

int bs_sched_refill(bs_sched* s, bs_sched_plan* plan) {
  if (!s || !plan) return sfail(BS_ERR_INVALID_ARG, "NULL argument");
  const bs_sched_config& c = s->cfg;
  s->admitted.clear();
  if (c.policy == BS_SCHED_FIXED) {
    while (!s->pending.empty() && (int)s->active.size() < c.fixed_batch && free_row(s) >= 0) take(s, 0);
  } else {
    for (;;) {
      // sand filling: candidates anywhere in the queue that do not widen the box
      int64_t box = 0;
      for (const SReq& r : s->active) box = std::max(box, r.width(c.L));
      for (size_t i = 0; i < s->pending.size() && free_row(s) >= 0;) {
        const SReq& q = s->pending[i];
        if ((int64_t)q.p + c.L <= box && eq1_cost(s, &q) <= c.budget)
          take(s, i);
        else
          ++i;
      }
      // then the head of the queue, if the enlarged set fits
      if (s->pending.empty() || free_row(s) < 0 || eq1_cost(s, &s->pending[0]) > c.budget) break;
      take(s, 0);
    }
  }
  // plan: descriptors in row order, K4 segments for the admitted requests
  std::vector<const SReq*> byrow;
  for (const SReq& r : s->active) byrow.push_back(&r);
  std::sort(byrow.begin(), byrow.end(), [](const SReq* x, const SReq* y) { return x->row < y->row; });
  s->descs.clear();
  s->ids.clear();
  for (const SReq* r : byrow) {
    s->descs.push_back(bs_req_desc{r->p, r->g, r->b, r->row, c.width - (r->p + r->g)});
    s->ids.push_back(r->id);
  }
  s->segs.clear();
  for (size_t a = 0; a < s->admitted.size(); ++a) {
    const SReq* r = nullptr;
    for (const SReq& x : s->active)
      if (x.id == s->admitted[a]) r = &x;
    const int len = r->p + r->g;
    s->segs.push_back(bs_copy_seg{1, (int32_t)a, 0, r->row, c.width - len, len});
  }
  int64_t box = 0;
  for (const SReq& r : s->active) box = std::max(box, r.width(c.L));
  plan->n_active = (int32_t)s->descs.size();
  plan->descs = s->descs.data();
  plan->ids = s->ids.data();
  plan->n_admitted = (int32_t)s->admitted.size();
  plan->admitted_ids = s->admitted.data();
  plan->segs = s->segs.data();
  plan->cost = eq1_cost(s, nullptr);
  plan->box_width = (int32_t)box;
  return BS_OK;
}

int bs_sched_complete(bs_sched* s, const uint8_t* eos, int n, int32_t* evicted_ids, int32_t* n_evicted) {
  if (!s || !n_evicted) return sfail(BS_ERR_INVALID_ARG, "NULL argument");
  if (n != (int)s->active.size()) return sfail(BS_ERR_INVALID_ARG, "n=%d but %zu requests are active", n, s->active.size());
  if (n > 0 && !evicted_ids) return sfail(BS_ERR_INVALID_ARG, "evicted_ids is NULL");
  const int L = s->cfg.L;
  // eos[] follows the row order of the last plan
  std::vector<const SReq*> byrow;
  for (const SReq& r : s->active) byrow.push_back(&r);
  std::sort(byrow.begin(), byrow.end(), [](const SReq* x, const SReq* y) { return x->row < y->row; });
  std::vector<int32_t> eos_ids;
  for (int i = 0; i < n; ++i)
    if (eos && eos[i]) eos_ids.push_back(byrow[i]->id);
  ++s->cycles;
  s->sum_active += n;
  int ne = 0;
  std::vector<SReq> keep;
  for (SReq r : s->active) {
    ++r.b;
    const bool e = std::find(eos_ids.begin(), eos_ids.end(), r.id) != eos_ids.end();
    if (r.b >= r.K(L) || e) {
      evicted_ids[ne++] = r.id;
      s->used[r.row] = 0;
      ++s->n_finished;
    } else {
      keep.push_back(r);
    }
  }
  s->active.swap(keep);
  *n_evicted = ne;
  return BS_OK;
}

int bs_sched_counts(const bs_sched* s, int32_t* n_pending, int32_t* n_active, int64_t* n_finished, int64_t* cycles,
                    int64_t* sum_active) {
  if (!s) return sfail(BS_ERR_INVALID_ARG, "scheduler is NULL");
  if (n_pending) *n_pending = (int32_t)s->pending.size();
  if (n_active) *n_active = (int32_t)s->active.size();
  if (n_finished) *n_finished = s->n_finished;
  if (cycles) *cycles = s->cycles;
  if (sum_active) *sum_active = s->sum_active;
  return BS_OK;
}

}  // extern "C"

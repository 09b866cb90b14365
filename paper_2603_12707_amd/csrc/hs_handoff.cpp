// hs_handoff.cpp — the aligned batch handoff between embedding arrival and
// language prefill (§5.2 "Aligned Batch Handoff": B_align = 32 by default and
// a 500 ms timeout; §5.3 "Parameter Sensitivity" discusses the choice of 32).
// Host logic only: requests whose
// projected embeddings have arrived wait in arrival order until a batch is
// due, and the batch goes to hs_prefill_batch.
#include <cmath>
#include <cstdint>
#include <deque>
#include <new>

#include "hs_internal.h"

struct hs_handoff {
  int align = 0;
  int64_t max_rows = 0;  // 0: no row budget
  int max_pending = 0;
  double timeout_ms = 0;
  struct Item {
    int32_t req;
    int32_t rows;
    double t;
  };
  std::deque<Item> pending;
};

namespace {

// The batch the queue would hand over now: the longest prefix of at most
// `align` requests whose rows fit the budget (at least one request).  *full
// tells whether it stopped on the budget with more requests waiting.
int candidate(const hs_handoff *h, int64_t *rows, bool *full) {
  int k = 0;
  int64_t r = 0;
  *full = false;
  for (const auto &it : h->pending) {
    if (k == h->align) break;
    if (k > 0 && h->max_rows > 0 && r + it.rows > h->max_rows) {
      *full = true;
      break;
    }
    r += it.rows;
    ++k;
  }
  *rows = r;
  return k;
}

}  // namespace

extern "C" {

int hs_handoff_create(int32_t align, int64_t max_rows, int32_t max_pending, double timeout_ms, hs_handoff **out) {
  if (!out) return hs::fail(HS_E_INVALID, "hs_handoff_create: out is NULL");
  *out = nullptr;
  if (align <= 0 || max_rows < 0 || max_pending < align || !(timeout_ms >= 0) || std::isinf(timeout_ms))
    return hs::fail(HS_E_INVALID, "hs_handoff_create: align %d, max_rows %lld, max_pending %d, timeout %g", align,
                    (long long)max_rows, max_pending, timeout_ms);
  hs_handoff *h = new (std::nothrow) hs_handoff();
  if (!h) return hs::fail(HS_E_DEVICE, "hs_handoff_create: out of host memory");
  h->align = align;
  h->max_rows = max_rows;
  h->max_pending = max_pending;
  h->timeout_ms = timeout_ms;
  *out = h;
  return HS_OK;
}

int hs_handoff_free(hs_handoff *h) {
  if (!h) return hs::fail(HS_E_INVALID, "hs_handoff_free: NULL");
  delete h;
  return HS_OK;
}

int hs_handoff_push(hs_handoff *h, int32_t req, int32_t rows, double now_ms) {
  if (!h) return hs::fail(HS_E_INVALID, "hs_handoff_push: NULL");
  if (req < 0 || rows <= 0 || !std::isfinite(now_ms))
    return hs::fail(HS_E_INVALID, "hs_handoff_push: request %d, rows %d", req, rows);
  if (!h->pending.empty() && now_ms < h->pending.back().t)
    return hs::fail(HS_E_INVALID, "hs_handoff_push: time %g before the last arrival %g", now_ms, h->pending.back().t);
  if ((int)h->pending.size() >= h->max_pending)
    return hs::fail(HS_E_CAPACITY, "hs_handoff_push: %d requests already wait", h->max_pending);
  h->pending.push_back({req, rows, now_ms});
  return HS_OK;
}

int hs_handoff_pop(hs_handoff *h, double now_ms, int32_t *reqs, int32_t max, int32_t *n, int64_t *rows,
                   double *wait_ms) {
  if (!h || !n) return hs::fail(HS_E_INVALID, "hs_handoff_pop: NULL");
  if (!std::isfinite(now_ms)) return hs::fail(HS_E_INVALID, "hs_handoff_pop: bad time");
  *n = 0;
  if (rows) *rows = 0;
  if (wait_ms) *wait_ms = -1;
  if (h->pending.empty()) return HS_OK;
  int64_t r;
  bool full;
  const int k = candidate(h, &r, &full);
  const double waited = now_ms - h->pending.front().t;
  const bool due = k == h->align || full || waited >= h->timeout_ms;
  if (!due) {
    if (wait_ms) *wait_ms = h->timeout_ms - waited;
    return HS_OK;
  }
  if (!reqs || max < k) return hs::fail(HS_E_BUFFER, "hs_handoff_pop: a batch of %d requests is due, room for %d", k, max);
  for (int i = 0; i < k; ++i) {
    reqs[i] = h->pending.front().req;
    h->pending.pop_front();
  }
  *n = k;
  if (rows) *rows = r;
  if (wait_ms && !h->pending.empty()) {
    int64_t r2;
    bool full2;
    const int k2 = candidate(h, &r2, &full2);
    *wait_ms = k2 == h->align || full2 ? 0.0 : std::fmax(0.0, h->timeout_ms - (now_ms - h->pending.front().t));
  }
  return HS_OK;
}

int hs_handoff_pending(const hs_handoff *h, int32_t *n) {
  if (!h || !n) return hs::fail(HS_E_INVALID, "hs_handoff_pending: NULL");
  *n = (int32_t)h->pending.size();
  return HS_OK;
}

}  // extern "C"

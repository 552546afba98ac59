// Greedy batch-size policy (Section 5.1, Algorithm "Inference") and its event-driven
// simulation over an arrival sequence.  Host code only; integer microseconds.
#include "greedy.h"

#include <algorithm>
#include <climits>
#include <vector>

namespace rafiki {

namespace {
constexpr int64_t kTimeLimit = int64_t(1) << 40;
constexpr int64_t kArrivalLimit = int64_t(1) << 61;

// Index of the largest candidate size <= queue_len, or -1.
int largest_fitting(const rafiki_greedy_policy& p, int64_t queue_len) {
  int j = -1;
  for (int i = 0; i < p.n_sizes; ++i)
    if (p.batch_sizes[i] <= queue_len) j = i;
  return j;
}
}  // namespace

int check_policy(const rafiki_greedy_policy* p) {
  if (!p || !p->batch_sizes || !p->cost_us) return set_error(RAFIKI_ERR_INVALID, "null policy or policy array");
  if (p->n_sizes < 1 || p->n_sizes > 64) return set_error(RAFIKI_ERR_INVALID, "n_sizes must be in [1, 64]");
  for (int i = 0; i < p->n_sizes; ++i) {
    if (p->batch_sizes[i] < 1 || (i > 0 && p->batch_sizes[i] <= p->batch_sizes[i - 1]))
      return set_error(RAFIKI_ERR_INVALID, "batch sizes must be >= 1 and strictly increasing");
    if (p->cost_us[i] < 0 || p->cost_us[i] >= kTimeLimit)
      return set_error(RAFIKI_ERR_INVALID, "batch costs must be in [0, 2^40) microseconds");
  }
  if (p->tau_us < 0 || p->tau_us >= kTimeLimit || p->delta_us < 0 || p->delta_us >= kTimeLimit)
    return set_error(RAFIKI_ERR_INVALID, "tau and delta must be in [0, 2^40) microseconds");
  return RAFIKI_OK;
}

int check_arrivals(const int64_t* a, int64_t n) {
  if (n < 0) return set_error(RAFIKI_ERR_INVALID, "n_requests must be >= 0");
  if (n > 0 && !a) return set_error(RAFIKI_ERR_INVALID, "null arrival array");
  for (int64_t i = 0; i < n; ++i) {
    if (a[i] < 0 || a[i] >= kArrivalLimit) return set_error(RAFIKI_ERR_INVALID, "arrival times must be in [0, 2^61)");
    if (i > 0 && a[i] < a[i - 1]) return set_error(RAFIKI_ERR_INVALID, "arrival times must be non-decreasing");
  }
  return RAFIKI_OK;
}

int32_t greedy_decide(const rafiki_greedy_policy& p, int64_t queue_len, int64_t oldest_wait_us) {
  const int32_t bmax = p.batch_sizes[p.n_sizes - 1];
  if (queue_len >= bmax) return bmax;
  const int j = largest_fitting(p, queue_len);
  if (j < 0) return 0;
  return p.cost_us[j] + oldest_wait_us + p.delta_us >= p.tau_us ? p.batch_sizes[j] : 0;
}

int64_t greedy_deadline(const rafiki_greedy_policy& p, int64_t queue_len, int64_t oldest_arrival_us) {
  const int j = largest_fitting(p, queue_len);
  if (j < 0) return INT64_MAX;
  return oldest_arrival_us + p.tau_us - p.delta_us - p.cost_us[j];
}

}  // namespace rafiki

using namespace rafiki;

extern "C" {

int rafiki_greedy_decide(const rafiki_greedy_policy* policy, int64_t queue_len, int64_t oldest_wait_us,
                         int32_t* out_b) {
  int rc = check_policy(policy);
  if (rc) return rc;
  if (!out_b) return set_error(RAFIKI_ERR_INVALID, "null out_b");
  if (queue_len < 0 || oldest_wait_us < 0 || oldest_wait_us >= kArrivalLimit)
    return set_error(RAFIKI_ERR_INVALID, "queue_len and oldest_wait_us must be >= 0");
  *out_b = greedy_decide(*policy, queue_len, oldest_wait_us);
  return RAFIKI_OK;
}

int rafiki_greedy_simulate(const rafiki_greedy_policy* policy, const int64_t* arrival_us, int64_t n_requests,
                           int64_t* out_latency_us, rafiki_dispatch* out_dispatch, int64_t dispatch_cap,
                           int64_t* out_n_dispatch) {
  int rc = check_policy(policy);
  if (!rc) rc = check_arrivals(arrival_us, n_requests);
  if (rc) return rc;
  if ((n_requests > 0 && !out_latency_us) || !out_n_dispatch || dispatch_cap < 0 ||
      (dispatch_cap > 0 && !out_dispatch))
    return set_error(RAFIKI_ERR_INVALID, "null output or negative dispatch_cap");
  const rafiki_greedy_policy& p = *policy;
  const int64_t* a = arrival_us;
  const int64_t n = n_requests;
  std::fill(out_latency_us, out_latency_us + n, int64_t(-1));
  int64_t nd = 0;
  int64_t t = n ? a[0] : 0;
  int64_t head = 0, arrived = 0;
  for (;;) {
    while (arrived < n && a[arrived] <= t) ++arrived;
    const int64_t qlen = arrived - head;
    if (qlen == 0) {
      if (arrived == n) break;
      t = a[arrived];
      continue;
    }
    const int64_t wait = t - a[head];
    const int32_t b = greedy_decide(p, qlen, wait);
    if (b > 0) {
      int64_t cost = 0;
      for (int i = 0; i < p.n_sizes; ++i)
        if (p.batch_sizes[i] == b) cost = p.cost_us[i];
      const int64_t done = t + cost;
      for (int64_t i = head; i < head + b; ++i) out_latency_us[i] = done - a[i];
      if (nd < dispatch_cap) out_dispatch[nd] = {t, done, head, qlen, wait, b, -1};
      ++nd;
      head += b;
      t = done;
      continue;
    }
    int64_t next = arrived < n ? a[arrived] : INT64_MAX;
    next = std::min(next, greedy_deadline(p, qlen, a[head]));
    if (next == INT64_MAX) break;     // below min(B) with no further arrivals
    t = next;
  }
  *out_n_dispatch = nd;
  return RAFIKI_OK;
}

int rafiki_greedy_simulate_multi(const rafiki_greedy_policy* policies, int n_servers, const int64_t* arrival_us,
                                 int64_t n_requests, int64_t* out_latency_us, rafiki_dispatch* out_dispatch,
                                 int64_t dispatch_cap, int64_t* out_n_dispatch) {
  if (!policies || n_servers < 1 || n_servers > 64)
    return set_error(RAFIKI_ERR_INVALID, "null policies or n_servers outside [1, 64]");
  for (int k = 0; k < n_servers; ++k)
    if (int rc = check_policy(&policies[k])) return rc;
  int rc = check_arrivals(arrival_us, n_requests);
  if (rc) return rc;
  if ((n_requests > 0 && !out_latency_us) || !out_n_dispatch || dispatch_cap < 0 ||
      (dispatch_cap > 0 && !out_dispatch))
    return set_error(RAFIKI_ERR_INVALID, "null output or negative dispatch_cap");
  const int64_t* a = arrival_us;
  const int64_t n = n_requests;
  std::fill(out_latency_us, out_latency_us + n, int64_t(-1));
  std::vector<int64_t> free_at(n_servers, INT64_MIN);
  int64_t nd = 0, t = n ? a[0] : 0, head = 0, arrived = 0;
  while (head < n) {
    while (arrived < n && a[arrived] <= t) ++arrived;
    // Free servers in index order, again until none dispatches: a dispatch changes the
    // queue's length and oldest request, which a server that declined before it must
    // see at the same instant (with costs that fall as b grows, it may now accept).
    for (bool again = true; again;) {
      again = false;
      for (int k = 0; k < n_servers; ++k) {
        if (free_at[k] > t || arrived == head) continue;
        const rafiki_greedy_policy& p = policies[k];
        const int64_t qlen = arrived - head, wait = t - a[head];
        const int32_t b = greedy_decide(p, qlen, wait);
        if (b == 0) continue;
        int64_t cost = 0;
        for (int i = 0; i < p.n_sizes; ++i)
          if (p.batch_sizes[i] == b) cost = p.cost_us[i];
        const int64_t done = t + cost;
        for (int64_t i = head; i < head + b; ++i) out_latency_us[i] = done - a[i];
        if (nd < dispatch_cap) out_dispatch[nd] = {t, done, head, qlen, wait, b, k};
        ++nd;
        head += b;
        free_at[k] = done;
        again = true;
      }
    }
    if (head >= n) break;
    int64_t next = arrived < n ? a[arrived] : INT64_MAX;
    for (int k = 0; k < n_servers; ++k) {
      if (free_at[k] > t) next = std::min(next, free_at[k]);
      else if (arrived > head) next = std::min(next, greedy_deadline(policies[k], arrived - head, a[head]));
    }
    if (next == INT64_MAX) break;   // nothing running, nothing servable, nothing arriving
    // every free server declined the final queue at t, so each deadline lies after t
    if (next <= t) return set_error(RAFIKI_ERR_INVALID, "internal: simulation clock did not advance");
    t = next;
  }
  *out_n_dispatch = nd;
  return RAFIKI_OK;
}

}  // extern "C"

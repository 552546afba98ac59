// Greedy batch-size policy shared by the host simulator and the real-time serving
// loops (internal to the library).
#pragma once
#include <cstdint>
#include <string>

#include "rafiki_sched.h"
#include "rafiki_rl.h"

namespace rafiki {

// Sets the thread's last-error text; returns code.
int set_error(int code, const std::string& msg);

// Validates a policy (RAFIKI_OK or RAFIKI_ERR_INVALID with the error text set).
int check_policy(const rafiki_greedy_policy* p);

// Algorithm "Inference" for one queue state: the batch size to serve now, or 0.
int32_t greedy_decide(const rafiki_greedy_policy& p, int64_t queue_len, int64_t oldest_wait_us);

// Earliest time at which waiting could end for a queue of queue_len >= min(B)
// requests whose oldest arrived at oldest_arrival_us: the instant its wait reaches
// tau - delta - c(b) for the largest fitting b.  Returns INT64_MAX below min(B).
int64_t greedy_deadline(const rafiki_greedy_policy& p, int64_t queue_len, int64_t oldest_arrival_us);

// Arrival times must be non-decreasing and in [0, 2^61).
int check_arrivals(const int64_t* a, int64_t n);

// The actor-critic scheduler's pieces used by the real-time serving loop.
struct RlAgentView {
  int n_models, n_sizes, queue_features, state_dim, n_actions;
  const int32_t* batch_sizes;
  int64_t tau_us;
};
RlAgentView rl_view(const rafiki_rl_s* h);
// The state of Section 5.2 from live quantities: waits [nq] of the queued requests
// (oldest first) and each model's time left on dispatched work busy_left [n_models].
void rl_live_state(const rafiki_rl_s* h, const int64_t* waits, int64_t nq, const int64_t* busy_left, double* s);
// mode 1: sample from the policy with one uniform draw of the splitmix64 stream *rng;
// mode 2: the most probable action (lowest index on ties).
int rl_choose(const rafiki_rl_s* h, const double* s, int mode, uint64_t* rng);
// Action index -> (subset mask, index into the batch sizes).
void rl_action(const rafiki_rl_s* h, int action, int* mask, int* size_index);

}  // namespace rafiki

// Greedy batch-size policy shared by the host simulator and the real-time serving
// loops (internal to the library).
#pragma once
#include <cstdint>
#include <string>

#include "rafiki_sched.h"

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

}  // namespace rafiki

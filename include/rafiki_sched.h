/*
 * rafiki_sched.h -- batch-size scheduling and request serving around the ensemble
 * (C ABI, MI355X / gfx950 library librafiki_ensemble.so).
 *
 * The paper serves a FIFO request queue with a greedy batch-size policy (Section 5.1,
 * Algorithm "Inference"): whenever the model is free, serve the oldest max(B)
 * requests if that many are queued; otherwise take b, the largest candidate size not
 * above the queue length, and serve the oldest b requests once
 * c(b) + w(q_0) + delta >= tau, where c(b) is the measured time of a batch of b,
 * w(q_0) the waiting time of the oldest queued request, tau the latency objective
 * and delta a back-off constant.  With fewer than min(B) requests queued it waits.
 * The objective it serves is Equation (single): the mean over all requests of
 * max(0, l(s) - tau), l(s) = waiting + inference time.
 *
 *   rafiki_greedy_decide     the policy's decision for one queue state
 *   rafiki_greedy_simulate   event-driven simulation of one model serving an arrival
 *                            sequence (host only; no device needed)
 *   rafiki_greedy_simulate_multi   the same for several independent servers sharing
 *                            the queue (one model each)
 *   rafiki_ensemble_profile  measures c(b) (or c(m, b)) on the device
 *   rafiki_ensemble_serve_greedy        real-time serving: every batch runs all
 *                            selected models and combines them (the synchronous
 *                            ensemble of Section 7.2)
 *   rafiki_ensemble_serve_greedy_async  real-time serving with each selected model an
 *                            independent server on its own stream, each batch served
 *                            by one model (the asynchronous, maximum-throughput
 *                            regime of Section 7.2)
 *
 * Conventions: times are integer microseconds; every function returns RAFIKI_OK or a
 * negative RAFIKI_ERR_* code (rafiki_ensemble.h) and sets rafiki_last_error().
 */
#ifndef RAFIKI_SCHED_H
#define RAFIKI_SCHED_H

#include <stdint.h>

#include "rafiki_ensemble.h"

#ifdef __cplusplus
extern "C" {
#endif

/* A greedy policy.  Host pointers, read during the call only.
 * batch_sizes: the candidate list B, strictly increasing, every entry >= 1.
 * cost_us:     c(b) for each candidate, in [0, 2^40).
 * n_sizes:     1..64.  tau_us, delta_us: in [0, 2^40).
 * Violations give RAFIKI_ERR_INVALID. */
typedef struct {
  const int32_t* batch_sizes;
  const int64_t* cost_us;
  int n_sizes;
  int64_t tau_us;
  int64_t delta_us;
} rafiki_greedy_policy;

/* One served batch.  Requests are served in arrival order, so a batch is the
 * contiguous request range [first, first + b). */
typedef struct {
  int64_t start_us;        /* decision time (simulation: the batch's start) */
  int64_t end_us;          /* completion time */
  int64_t first;           /* index of the batch's oldest request */
  int64_t queue_len;       /* queue length seen by the decision */
  int64_t oldest_wait_us;  /* w(q_0) seen by the decision */
  int32_t b;               /* batch size */
  int32_t model;           /* serving model (asynchronous serving), -1 for an ensemble */
} rafiki_dispatch;

/* *out_b = the batch size to serve now, or 0 to keep waiting, for a queue of
 * queue_len >= 0 requests whose oldest has waited oldest_wait_us. */
int rafiki_greedy_decide(const rafiki_greedy_policy* policy, int64_t queue_len, int64_t oldest_wait_us,
                         int32_t* out_b);

/* Simulate one model serving requests that arrive at arrival_us[0..n_requests)
 * (non-decreasing, in [0, 2^61)).  The model starts free at arrival_us[0]; a batch
 * started at t ends at t + c(b), and the decision is re-taken exactly when a request
 * arrives, the model becomes free, or the oldest request's wait reaches
 * tau - delta - c(b).
 * out_latency_us [n_requests] (host): completion time minus arrival time, or -1 for a
 * request never served (fewer than min(B) requests left with no further arrivals).
 * out_dispatch (host, may be NULL when dispatch_cap == 0): the first dispatch_cap
 * batches; *out_n_dispatch = the total number of batches (which may exceed the cap). */
int rafiki_greedy_simulate(const rafiki_greedy_policy* policy, const int64_t* arrival_us, int64_t n_requests,
                           int64_t* out_latency_us, rafiki_dispatch* out_dispatch, int64_t dispatch_cap,
                           int64_t* out_n_dispatch);

/* Simulate n_servers independent servers (for example one model each) sharing one
 * FIFO queue: whenever a server is free (servers visited in index order), the greedy
 * policy policies[k] (its own c(b)) decides a batch of the oldest queued requests for
 * it.  Decisions are re-taken exactly when a request arrives, a server becomes free
 * or a free server's deadline is reached.  Outputs as rafiki_greedy_simulate; each
 * dispatch's `model` is its server.  n_servers in [1, 64].  This is the host model of
 * rafiki_ensemble_serve_greedy_async with c(m, b) as given. */
int rafiki_greedy_simulate_multi(const rafiki_greedy_policy* policies, int n_servers, const int64_t* arrival_us,
                                 int64_t n_requests, int64_t* out_latency_us, rafiki_dispatch* out_dispatch,
                                 int64_t dispatch_cap, int64_t* out_n_dispatch);

/* Measure c(b) on the device: for every candidate b (1 <= b <= max_batch), the median
 * over `reps` (1..1000) timed runs of rafiki_ensemble_infer(h, batch, b, mask, ...)
 * after one untimed run, timed with HIP events on `stream`; rounded up to whole
 * microseconds into out_cost_us[n_sizes] (host).  `batch` holds at least max(B)
 * requests (device, opts.input_kind layout); `scratch_probs` (device fp32
 * [max(B), n_classes]) and `scratch_labels` (device int32 [max(B)]) receive the
 * outputs.  mask = 1 << m gives c(m, b).  Blocks the caller. */
int rafiki_ensemble_profile(rafiki_ensemble_t h, const void* batch, const int32_t* batch_sizes, int n_sizes,
                            uint32_t mask, int reps, float* scratch_probs, int32_t* scratch_labels,
                            int64_t* out_cost_us, void* stream);

/* Serve requests in real time with the greedy policy.  Request i is row i of
 * `requests` (device, opts.input_kind layout, n_requests rows, all resident before
 * the call) and arrives arrival_us[i] microseconds after the call starts serving
 * (non-decreasing host array).  Before the clock starts, every candidate size is run
 * once (this also tunes the kernels for it).  Each batch runs rafiki_ensemble_infer
 * (combine = 0) or rafiki_ensemble_infer_vote (combine = 1) with `mask` on rows
 * [first, first + b) and writes out_probs rows [first, first + b) (device fp32
 * [n_requests, n_classes]) and out_labels (device int32 [n_requests]); the host waits
 * for the batch to finish before the next decision.  out_latency_us [n_requests]
 * (host) receives completion minus arrival time, or -1 for requests never served;
 * out_dispatch / *out_n_dispatch as in rafiki_greedy_simulate.  Blocks the caller
 * until every servable request is done.  Requires max(B) <= max_batch. */
int rafiki_ensemble_serve_greedy(rafiki_ensemble_t h, const void* requests, const int64_t* arrival_us,
                                 int64_t n_requests, const rafiki_greedy_policy* policy, uint32_t mask,
                                 int combine, float* out_probs, int32_t* out_labels, int64_t* out_latency_us,
                                 rafiki_dispatch* out_dispatch, int64_t dispatch_cap, int64_t* out_n_dispatch,
                                 void* stream);

/* Serve requests in real time with every model selected by `mask` acting as an
 * independent server on its own stream: whenever a selected model is free (models
 * visited in index order), the greedy policy policies[m] (its own c(m, b)) decides a
 * batch of the oldest queued requests for it, and that batch's output rows are model
 * m's softmax probabilities and first-index argmax (no ensemble).  `policies` has
 * n_models entries; entries of unselected models are ignored.  Other arguments as
 * rafiki_ensemble_serve_greedy.
 * Image inputs get a staging buffer per model (allocated on the first call). */
int rafiki_ensemble_serve_greedy_async(rafiki_ensemble_t h, const void* requests, const int64_t* arrival_us,
                                       int64_t n_requests, const rafiki_greedy_policy* policies, uint32_t mask,
                                       float* out_probs, int32_t* out_labels, int64_t* out_latency_us,
                                       rafiki_dispatch* out_dispatch, int64_t dispatch_cap, int64_t* out_n_dispatch,
                                       void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RAFIKI_SCHED_H */

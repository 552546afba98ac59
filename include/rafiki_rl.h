/*
 * rafiki_rl.h -- reinforcement-learning scheduler for ensemble serving (C ABI, host
 * code in librafiki_ensemble.so).
 *
 * With several models the paper trades accuracy against latency by choosing, for each
 * batch, both the batch size and the subset of models that serve it, with an
 * actor-critic agent (Section 5.2):
 *   state   the waiting times of the queued requests (zero-padded or truncated to a
 *           fixed length), then the model status: c(m, b) for every model and
 *           candidate size, and each model's time left on the work dispatched to it;
 *   action  (v, b): a non-empty model mask v and a batch size b from B, i.e.
 *           (2^|M| - 1) * |B| actions, indexed mask-major (mask 1 .. 2^|M| - 1, then b);
 *   reward  a(M[v]) * (b - beta * |{s in batch : l(s) > tau}|) (Equation
 *           multi_acc_reward), a(M[v]) the surrogate accuracy of the ensemble v.
 *
 * Environment: each model is an independent server (one model per node or GPU).  A
 * decision is taken whenever requests are queued and at least one model is free; the
 * batch is the oldest min(b, queue length) requests; it starts on model m when m is
 * free, occupies it for c(m, b) and completes when its last model finishes; a
 * request's latency is completion minus arrival.  Times are integer microseconds;
 * state features are divided by tau.
 *
 * Agent: two tanh hidden layers of width H shared by a softmax policy head and a
 * linear value head; parameters (float64) are laid out W1 [H][D], b1 [H], W2 [H][H],
 * b2 [H], Wp [A][H], bp [A], Wv [1][H], bv [1].  Loss over T transitions
 *   (1/T) sum_t [ -log pi(a_t|s_t) A_t + c_v (V(s_t) - R_t)^2 - c_e H(pi(.|s_t)) ],
 * A_t = R_t - V(s_t) held constant; Adam updates (beta1 0.9, beta2 0.999, eps 1e-8).
 *
 * All functions return RAFIKI_OK or a negative RAFIKI_ERR_* code (rafiki_ensemble.h)
 * and set rafiki_last_error(); all pointers are host pointers read or written during
 * the call only.  A handle is not safe for concurrent use from several threads.
 */
#ifndef RAFIKI_RL_H
#define RAFIKI_RL_H

#include <stdint.h>

#include "rafiki_ensemble.h"
#include "rafiki_sched.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int n_models;                 /* 1..8 */
  const int32_t* batch_sizes;   /* B: strictly increasing, >= 1 */
  int n_sizes;                  /* 1..16 */
  const int64_t* cost_us;       /* [n_models * n_sizes]: c(m, B[j]) at m * n_sizes + j, in [1, 2^40) */
  const double* accuracy;       /* [1 << n_models]: a(M[v]) at index v (index 0 unused) */
  int64_t tau_us;               /* latency objective, in [1, 2^40) */
  double beta;                  /* weight of overdue requests in the reward, >= 0 */
  int queue_features;           /* number of waiting-time features, 1..4096 */
  int hidden;                   /* hidden width, 1..1024 */
} rafiki_rl_config;

typedef struct rafiki_rl_s* rafiki_rl_t;

/* Create an agent; parameters drawn uniformly in +-1/sqrt(fan-in) (policy head scaled
 * by 0.01) from a splitmix64 stream seeded with `seed`; Adam moments zero. */
int rafiki_rl_create(const rafiki_rl_config* cfg, uint64_t seed, rafiki_rl_t* out);
int rafiki_rl_destroy(rafiki_rl_t h);   /* NULL accepted */

/* State dimension D = queue_features + n_models * n_sizes + n_models, number of
 * actions A, number of parameters. */
int rafiki_rl_info(rafiki_rl_t h, int* state_dim, int* n_actions, int64_t* n_params);

/* Copy the parameters out / in (n must equal the parameter count); set also resets
 * the Adam moments and step counter. */
int rafiki_rl_get_params(rafiki_rl_t h, double* out, int64_t n);
int rafiki_rl_set_params(rafiki_rl_t h, const double* in, int64_t n);

/* Policy probabilities out_pi [A] and value *out_value of one state [D]. */
int rafiki_rl_forward(rafiki_rl_t h, const double* state, double* out_pi, double* out_value);

/* Gradient [n_params] of the loss above over T >= 1 transitions: states [T][D],
 * actions [T] in [0, A), returns [T]. */
int rafiki_rl_gradient(rafiki_rl_t h, const double* states, const int32_t* actions, const double* returns,
                       int64_t T, double c_v, double c_e, double* out_grad);

/* One Adam step with learning rate lr on the given gradient [n_params]. */
int rafiki_rl_adam_step(rafiki_rl_t h, const double* grad, double lr);

/* Run one episode over requests arriving at arrival_us[0..n) (non-decreasing).
 * mode 0: take actions_in[k] at decision k (the episode ends early if actions_in runs
 *         out: *out_steps < decisions needed);
 * mode 1: sample each action from the policy (splitmix64 stream seeded with `seed`);
 * mode 2: take the policy's most probable action (lowest index on ties).
 * Outputs (any may be NULL when cap == 0, except out_steps): out_actions [cap],
 * out_rewards [cap], out_states [cap][D], out_times [cap] (decision instants), the
 * number of decisions *out_steps, and out_latency [n] (-1 for requests not served). */
int rafiki_rl_run_episode(rafiki_rl_t h, const int64_t* arrival_us, int64_t n, int mode, const int32_t* actions_in,
                          int64_t n_actions_in, uint64_t seed, int32_t* out_actions, double* out_rewards,
                          double* out_states, int64_t* out_times, int64_t cap, int64_t* out_steps,
                          int64_t* out_latency);

/* Train with the actor-critic loss: `episodes` sampled episodes over the same arrival
 * sequence (episode e samples with seed + e); after each, returns R_t are the
 * discounted sums (factor gamma) of the rewards divided by max(B), and one Adam step
 * of rate lr is taken on the gradient over the episode's transitions.
 * out_episode_reward [episodes] (may be NULL) receives each episode's total reward. */
int rafiki_rl_train(rafiki_rl_t h, const int64_t* arrival_us, int64_t n, int episodes, double gamma, double lr,
                    double c_v, double c_e, uint64_t seed, double* out_episode_reward);

/* Serve requests in real time with the agent choosing each batch (Section 5.2): at
 * every decision the state is built from the live queue (the waits of the oldest
 * queued requests at that instant, the agent's c(m, b) table, each model's time left),
 * the agent picks (v, b) (mode 1: sampled with the splitmix64 stream seeded with
 * `seed`, one uniform draw per decision; mode 2: the most probable action, lowest index
 * on ties), and the oldest min(b, queue length) requests run through
 * rafiki_ensemble_infer with mask v on `stream`; their output rows go to out_probs /
 * out_labels (device, [n_requests, n_classes] / [n_requests]).  The selected models of
 * a batch run concurrently on the one GPU inside that call and the host waits for it
 * to complete before the next decision, so every decision sees all models free (the
 * time-left features are zero).  Request i is row i of `requests` (device, resident
 * before the call) and arrives arrival_us[i] microseconds after serving starts (host,
 * non-decreasing).  Before the clock starts every subset runs once at every batch
 * size from 1 to max(B), the sizes min(b, queue length) can take (tuning).  Logs (host, first `cap` decisions): out_dispatch[k] (start = the
 * decision instant, end, first request, queue length, oldest wait, batch size served,
 * model -1), out_actions[k] and out_states[k * state_dim ...]; *out_steps = the number
 * of decisions.  out_latency_us[n_requests] (host) = completion minus arrival.  The
 * agent must schedule n_models models and its largest size must not exceed max_batch
 * (else RAFIKI_ERR_INVALID).  Blocks the caller until every request is served. */
int rafiki_ensemble_serve_rl(rafiki_ensemble_t h, rafiki_rl_t agent, const void* requests, const int64_t* arrival_us,
                             int64_t n_requests, int mode, uint64_t seed, float* out_probs, int32_t* out_labels,
                             int64_t* out_latency_us, rafiki_dispatch* out_dispatch, int32_t* out_actions,
                             double* out_states, int64_t cap, int64_t* out_steps, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RAFIKI_RL_H */

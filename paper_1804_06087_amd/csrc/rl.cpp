// Actor-critic scheduler for ensemble serving (Section 5.2): environment, two-layer
// tanh policy / value network with hand-written backpropagation, Adam, episode
// rollout and training.  Host code, float64.
#include "rafiki_rl.h"

#include "greedy.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <memory>
#include <string>
#include <vector>

using namespace rafiki;

namespace {

constexpr int64_t kTimeLimit = int64_t(1) << 40;

// splitmix64 (Steele, Lea and Flood): a counter-based 64-bit generator.
struct SplitMix {
  uint64_t x;
  uint64_t next() {
    uint64_t z = (x += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
  double uniform() { return (double)(next() >> 11) * (1.0 / 9007199254740992.0); }   // [0, 1)
};

struct Layout {   // offsets of the parameter blocks
  int D, H, A;
  int64_t W1, b1, W2, b2, Wp, bp, Wv, bv, n;
  void init(int D_, int H_, int A_) {
    D = D_; H = H_; A = A_;
    int64_t k = 0;
    W1 = k; k += (int64_t)H * D;
    b1 = k; k += H;
    W2 = k; k += (int64_t)H * H;
    b2 = k; k += H;
    Wp = k; k += (int64_t)A * H;
    bp = k; k += A;
    Wv = k; k += H;
    bv = k; k += 1;
    n = k;
  }
};

// Forward pass keeping the activations for backpropagation.
struct Acts {
  std::vector<double> h1, h2, pi;
  double v = 0;
};

void forward(const Layout& L, const double* th, const double* s, Acts& o) {
  o.h1.assign(L.H, 0.0);
  o.h2.assign(L.H, 0.0);
  o.pi.assign(L.A, 0.0);
  for (int i = 0; i < L.H; ++i) {
    double z = th[L.b1 + i];
    const double* w = th + L.W1 + (int64_t)i * L.D;
    for (int j = 0; j < L.D; ++j) z += w[j] * s[j];
    o.h1[i] = std::tanh(z);
  }
  for (int i = 0; i < L.H; ++i) {
    double z = th[L.b2 + i];
    const double* w = th + L.W2 + (int64_t)i * L.H;
    for (int j = 0; j < L.H; ++j) z += w[j] * o.h1[j];
    o.h2[i] = std::tanh(z);
  }
  double zmax = -INFINITY;
  for (int a = 0; a < L.A; ++a) {
    double z = th[L.bp + a];
    const double* w = th + L.Wp + (int64_t)a * L.H;
    for (int j = 0; j < L.H; ++j) z += w[j] * o.h2[j];
    o.pi[a] = z;
    zmax = std::max(zmax, z);
  }
  double sum = 0;
  for (int a = 0; a < L.A; ++a) {
    o.pi[a] = std::exp(o.pi[a] - zmax);
    sum += o.pi[a];
  }
  for (int a = 0; a < L.A; ++a) o.pi[a] /= sum;
  double v = th[L.bv];
  for (int j = 0; j < L.H; ++j) v += th[L.Wv + j] * o.h2[j];
  o.v = v;
}

// Accumulate the loss gradient of one transition into g (not yet divided by T).
void backward(const Layout& L, const double* th, const double* s, int act, double ret, double c_v, double c_e,
              const Acts& o, double* g, std::vector<double>& dz, std::vector<double>& dh) {
  const double adv = ret - o.v;
  double ent = 0;
  for (int a = 0; a < L.A; ++a) ent -= o.pi[a] * std::log(o.pi[a]);
  dz.resize(L.A);
  for (int a = 0; a < L.A; ++a) {
    dz[a] = (o.pi[a] - (a == act ? 1.0 : 0.0)) * adv + c_e * o.pi[a] * (std::log(o.pi[a]) + ent);
  }
  const double dv = 2.0 * c_v * (o.v - ret);
  dh.assign(2 * L.H, 0.0);
  double* dh2 = dh.data();
  double* dh1 = dh.data() + L.H;
  for (int a = 0; a < L.A; ++a) {
    g[L.bp + a] += dz[a];
    double* gw = g + L.Wp + (int64_t)a * L.H;
    const double* w = th + L.Wp + (int64_t)a * L.H;
    for (int j = 0; j < L.H; ++j) {
      gw[j] += dz[a] * o.h2[j];
      dh2[j] += w[j] * dz[a];
    }
  }
  g[L.bv] += dv;
  for (int j = 0; j < L.H; ++j) {
    g[L.Wv + j] += dv * o.h2[j];
    dh2[j] += dv * th[L.Wv + j];
  }
  for (int i = 0; i < L.H; ++i) {
    const double da = dh2[i] * (1.0 - o.h2[i] * o.h2[i]);
    g[L.b2 + i] += da;
    double* gw = g + L.W2 + (int64_t)i * L.H;
    const double* w = th + L.W2 + (int64_t)i * L.H;
    for (int j = 0; j < L.H; ++j) {
      gw[j] += da * o.h1[j];
      dh1[j] += w[j] * da;
    }
  }
  for (int i = 0; i < L.H; ++i) {
    const double da = dh1[i] * (1.0 - o.h1[i] * o.h1[i]);
    g[L.b1 + i] += da;
    double* gw = g + L.W1 + (int64_t)i * L.D;
    for (int j = 0; j < L.D; ++j) gw[j] += da * s[j];
  }
}

}  // namespace

struct rafiki_rl_s {
  int M = 0, nB = 0, Lq = 0, H = 0, A = 0, D = 0;
  std::vector<int32_t> B;
  std::vector<int64_t> cost;   // [M][nB]
  std::vector<double> acc;     // [1 << M]
  int64_t tau = 1;
  double beta = 0;
  Layout lay;
  std::vector<double> theta, m1, m2;
  int64_t adam_t = 0;
  std::vector<int> act_mask, act_j;   // action -> (mask, size index)
};

namespace {

// The environment of Section 5.2 (see the header).
struct Env {
  const rafiki_rl_s* h;
  const int64_t* a;
  int64_t n, t = 0, head = 0, arrived = 0;
  std::vector<int64_t> busy;
  int64_t* lat;

  Env(const rafiki_rl_s* h_, const int64_t* a_, int64_t n_, int64_t* lat_) : h(h_), a(a_), n(n_), lat(lat_) {
    busy.assign(h->M, 0);
    t = n ? a[0] : 0;
    if (lat) std::fill(lat, lat + n, int64_t(-1));
    advance();
  }
  bool done() const { return head >= n; }
  void advance() {
    while (head < n) {
      while (arrived < n && a[arrived] <= t) ++arrived;
      const int64_t free = *std::min_element(busy.begin(), busy.end());
      if (arrived == head) {
        t = std::max(a[arrived], t);
        continue;
      }
      if (free > t) {
        t = free;
        continue;
      }
      return;
    }
  }
  void state(double* s) const {
    const double tau = (double)h->tau;
    int k = 0;
    for (int64_t i = head; i < std::min(arrived, head + h->Lq); ++i) s[k++] = (double)(t - a[i]) / tau;
    while (k < h->Lq) s[k++] = 0.0;
    for (int64_t c : h->cost) s[k++] = (double)c / tau;
    for (int m = 0; m < h->M; ++m) s[k++] = (double)std::max<int64_t>(busy[m] - t, 0) / tau;
  }
  double step(int action) {
    const int mask = h->act_mask[action], j = h->act_j[action];
    const int64_t nb = std::min<int64_t>(h->B[j], arrived - head);
    int64_t end = 0;
    for (int m = 0; m < h->M; ++m)
      if ((mask >> m) & 1) {
        const int64_t e = std::max(t, busy[m]) + h->cost[(size_t)m * h->nB + j];
        busy[m] = e;
        end = std::max(end, e);
      }
    int64_t over = 0;
    for (int64_t i = head; i < head + nb; ++i) {
      const int64_t l = end - a[i];
      if (lat) lat[i] = l;
      over += l > h->tau ? 1 : 0;
    }
    head += nb;
    advance();
    return h->acc[mask] * ((double)nb - h->beta * (double)over);
  }
};

int check_handle(rafiki_rl_t h) { return h ? RAFIKI_OK : set_error(RAFIKI_ERR_INVALID, "null handle"); }

// One action of the policy at state s (mode 1: sampled with the uniform draw u; mode 2:
// the most probable, lowest index on ties).
int pick_action(const rafiki_rl_s* h, const Acts& o, int mode, double u) {
  if (mode == 2) return (int)(std::max_element(o.pi.begin(), o.pi.end()) - o.pi.begin());
  double c = 0;
  for (int i = 0; i < h->A; ++i) {
    c += o.pi[i];
    if (u < c) return i;
  }
  return h->A - 1;
}

}  // namespace

namespace rafiki {

RlAgentView rl_view(const rafiki_rl_s* h) {
  return {h->M, h->nB, h->Lq, h->D, h->A, h->B.data(), h->tau};
}

void rl_live_state(const rafiki_rl_s* h, const int64_t* waits, int64_t nq, const int64_t* busy_left, double* s) {
  const double tau = (double)h->tau;
  int k = 0;
  for (int64_t i = 0; i < std::min<int64_t>(nq, h->Lq); ++i) s[k++] = (double)waits[i] / tau;
  while (k < h->Lq) s[k++] = 0.0;
  for (int64_t c : h->cost) s[k++] = (double)c / tau;
  for (int m = 0; m < h->M; ++m) s[k++] = (double)std::max<int64_t>(busy_left[m], 0) / tau;
}

int rl_choose(const rafiki_rl_s* h, const double* s, int mode, uint64_t* rng) {
  Acts o;
  forward(h->lay, h->theta.data(), s, o);
  double u = 0.0;
  if (mode == 1) {
    SplitMix r{*rng};
    u = r.uniform();
    *rng = r.x;
  }
  return pick_action(h, o, mode, u);
}

void rl_action(const rafiki_rl_s* h, int action, int* mask, int* size_index) {
  *mask = h->act_mask[action];
  *size_index = h->act_j[action];
}

}  // namespace rafiki

extern "C" {

int rafiki_rl_create(const rafiki_rl_config* c, uint64_t seed, rafiki_rl_t* out) {
  if (out) *out = nullptr;
  if (!c || !out) return set_error(RAFIKI_ERR_INVALID, "null argument");
  if (c->n_models < 1 || c->n_models > 8) return set_error(RAFIKI_ERR_INVALID, "n_models must be in [1, 8]");
  if (c->n_sizes < 1 || c->n_sizes > 16 || !c->batch_sizes || !c->cost_us || !c->accuracy)
    return set_error(RAFIKI_ERR_INVALID, "n_sizes must be in [1, 16] and the arrays non-null");
  for (int j = 0; j < c->n_sizes; ++j)
    if (c->batch_sizes[j] < 1 || (j && c->batch_sizes[j] <= c->batch_sizes[j - 1]))
      return set_error(RAFIKI_ERR_INVALID, "batch sizes must be >= 1 and strictly increasing");
  for (int i = 0; i < c->n_models * c->n_sizes; ++i)
    if (c->cost_us[i] < 1 || c->cost_us[i] >= kTimeLimit)
      return set_error(RAFIKI_ERR_INVALID, "costs must be in [1, 2^40) microseconds");
  for (int v = 1; v < (1 << c->n_models); ++v)
    if (!std::isfinite(c->accuracy[v])) return set_error(RAFIKI_ERR_INVALID, "accuracies must be finite");
  if (c->tau_us < 1 || c->tau_us >= kTimeLimit || !(c->beta >= 0) || !std::isfinite(c->beta))
    return set_error(RAFIKI_ERR_INVALID, "tau must be in [1, 2^40) and beta finite and >= 0");
  if (c->queue_features < 1 || c->queue_features > 4096 || c->hidden < 1 || c->hidden > 1024)
    return set_error(RAFIKI_ERR_INVALID, "queue_features must be in [1, 4096] and hidden in [1, 1024]");
  std::unique_ptr<rafiki_rl_s> h(new rafiki_rl_s);
  h->M = c->n_models;
  h->nB = c->n_sizes;
  h->Lq = c->queue_features;
  h->H = c->hidden;
  h->B.assign(c->batch_sizes, c->batch_sizes + c->n_sizes);
  h->cost.assign(c->cost_us, c->cost_us + (size_t)c->n_models * c->n_sizes);
  h->acc.assign(c->accuracy, c->accuracy + (1 << c->n_models));
  h->acc[0] = 0.0;
  h->tau = c->tau_us;
  h->beta = c->beta;
  for (int v = 1; v < (1 << h->M); ++v)
    for (int j = 0; j < h->nB; ++j) {
      h->act_mask.push_back(v);
      h->act_j.push_back(j);
    }
  h->A = (int)h->act_mask.size();
  h->D = h->Lq + h->M * h->nB + h->M;
  h->lay.init(h->D, h->H, h->A);
  h->theta.assign(h->lay.n, 0.0);
  SplitMix rng{seed};
  auto fill = [&](int64_t off, int64_t count, double bound) {
    for (int64_t i = 0; i < count; ++i) h->theta[off + i] = (2.0 * rng.uniform() - 1.0) * bound;
  };
  const Layout& L = h->lay;
  fill(L.W1, (int64_t)L.H * L.D, 1.0 / std::sqrt((double)L.D));
  fill(L.b1, L.H, 1.0 / std::sqrt((double)L.D));
  fill(L.W2, (int64_t)L.H * L.H, 1.0 / std::sqrt((double)L.H));
  fill(L.b2, L.H, 1.0 / std::sqrt((double)L.H));
  fill(L.Wp, (int64_t)L.A * L.H, 0.01 / std::sqrt((double)L.H));
  fill(L.bp, L.A, 0.0);
  fill(L.Wv, L.H, 1.0 / std::sqrt((double)L.H));
  fill(L.bv, 1, 0.0);
  h->m1.assign(L.n, 0.0);
  h->m2.assign(L.n, 0.0);
  *out = h.release();
  return RAFIKI_OK;
}

int rafiki_rl_destroy(rafiki_rl_t h) {
  delete h;
  return RAFIKI_OK;
}

int rafiki_rl_info(rafiki_rl_t h, int* state_dim, int* n_actions, int64_t* n_params) {
  if (int rc = check_handle(h)) return rc;
  if (state_dim) *state_dim = h->D;
  if (n_actions) *n_actions = h->A;
  if (n_params) *n_params = h->lay.n;
  return RAFIKI_OK;
}

int rafiki_rl_get_params(rafiki_rl_t h, double* out, int64_t n) {
  if (int rc = check_handle(h)) return rc;
  if (!out || n != h->lay.n) return set_error(RAFIKI_ERR_INVALID, "parameter buffer missing or of the wrong size");
  std::memcpy(out, h->theta.data(), sizeof(double) * n);
  return RAFIKI_OK;
}

int rafiki_rl_set_params(rafiki_rl_t h, const double* in, int64_t n) {
  if (int rc = check_handle(h)) return rc;
  if (!in || n != h->lay.n) return set_error(RAFIKI_ERR_INVALID, "parameter buffer missing or of the wrong size");
  for (int64_t i = 0; i < n; ++i)
    if (!std::isfinite(in[i])) return set_error(RAFIKI_ERR_INVALID, "parameters must be finite");
  std::memcpy(h->theta.data(), in, sizeof(double) * n);
  std::fill(h->m1.begin(), h->m1.end(), 0.0);
  std::fill(h->m2.begin(), h->m2.end(), 0.0);
  h->adam_t = 0;
  return RAFIKI_OK;
}

int rafiki_rl_forward(rafiki_rl_t h, const double* state, double* out_pi, double* out_value) {
  if (int rc = check_handle(h)) return rc;
  if (!state || !out_pi || !out_value) return set_error(RAFIKI_ERR_INVALID, "null argument");
  Acts o;
  forward(h->lay, h->theta.data(), state, o);
  std::copy(o.pi.begin(), o.pi.end(), out_pi);
  *out_value = o.v;
  return RAFIKI_OK;
}

int rafiki_rl_gradient(rafiki_rl_t h, const double* states, const int32_t* actions, const double* returns,
                       int64_t T, double c_v, double c_e, double* out_grad) {
  if (int rc = check_handle(h)) return rc;
  if (T < 1 || !states || !actions || !returns || !out_grad)
    return set_error(RAFIKI_ERR_INVALID, "T must be >= 1 and the arrays non-null");
  for (int64_t t = 0; t < T; ++t)
    if (actions[t] < 0 || actions[t] >= h->A) return set_error(RAFIKI_ERR_INVALID, "action out of range");
  std::fill(out_grad, out_grad + h->lay.n, 0.0);
  Acts o;
  std::vector<double> dz, dh;
  for (int64_t t = 0; t < T; ++t) {
    const double* s = states + t * h->D;
    forward(h->lay, h->theta.data(), s, o);
    backward(h->lay, h->theta.data(), s, actions[t], returns[t], c_v, c_e, o, out_grad, dz, dh);
  }
  for (int64_t i = 0; i < h->lay.n; ++i) out_grad[i] /= (double)T;
  return RAFIKI_OK;
}

int rafiki_rl_adam_step(rafiki_rl_t h, const double* g, double lr) {
  if (int rc = check_handle(h)) return rc;
  if (!g || !(lr > 0) || !std::isfinite(lr)) return set_error(RAFIKI_ERR_INVALID, "null gradient or bad rate");
  const double b1 = 0.9, b2 = 0.999, eps = 1e-8;
  ++h->adam_t;
  const double c1 = 1.0 - std::pow(b1, (double)h->adam_t), c2 = 1.0 - std::pow(b2, (double)h->adam_t);
  for (int64_t i = 0; i < h->lay.n; ++i) {
    h->m1[i] = b1 * h->m1[i] + (1 - b1) * g[i];
    h->m2[i] = b2 * h->m2[i] + (1 - b2) * g[i] * g[i];
    h->theta[i] -= lr * (h->m1[i] / c1) / (std::sqrt(h->m2[i] / c2) + eps);
  }
  return RAFIKI_OK;
}

int rafiki_rl_run_episode(rafiki_rl_t h, const int64_t* arrival_us, int64_t n, int mode, const int32_t* actions_in,
                          int64_t n_actions_in, uint64_t seed, int32_t* out_actions, double* out_rewards,
                          double* out_states, int64_t* out_times, int64_t cap, int64_t* out_steps,
                          int64_t* out_latency) {
  if (int rc = check_handle(h)) return rc;
  if (int rc = check_arrivals(arrival_us, n)) return rc;
  if (mode < 0 || mode > 2 || !out_steps || cap < 0 || (mode == 0 && n_actions_in > 0 && !actions_in))
    return set_error(RAFIKI_ERR_INVALID, "bad mode, cap or action list");
  if (mode == 0)
    for (int64_t k = 0; k < n_actions_in; ++k)
      if (actions_in[k] < 0 || actions_in[k] >= h->A) return set_error(RAFIKI_ERR_INVALID, "action out of range");
  Env env(h, arrival_us, n, out_latency);
  SplitMix rng{seed};
  std::vector<double> s(h->D);
  Acts o;
  int64_t k = 0;
  while (!env.done()) {
    if (mode == 0 && k >= n_actions_in) break;
    env.state(s.data());
    int act;
    if (mode == 0) {
      act = actions_in[k];
    } else {
      forward(h->lay, h->theta.data(), s.data(), o);
      act = pick_action(h, o, mode, mode == 1 ? rng.uniform() : 0.0);
    }
    const int64_t t0 = env.t;
    const double r = env.step(act);
    if (k < cap) {
      if (out_actions) out_actions[k] = act;
      if (out_rewards) out_rewards[k] = r;
      if (out_states) std::copy(s.begin(), s.end(), out_states + k * h->D);
      if (out_times) out_times[k] = t0;
    }
    ++k;
  }
  *out_steps = k;
  return RAFIKI_OK;
}

int rafiki_rl_train(rafiki_rl_t h, const int64_t* arrival_us, int64_t n, int episodes, double gamma, double lr,
                    double c_v, double c_e, uint64_t seed, double* out_episode_reward) {
  if (int rc = check_handle(h)) return rc;
  if (int rc = check_arrivals(arrival_us, n)) return rc;
  if (n < 1 || episodes < 1 || !(gamma >= 0 && gamma <= 1) || !(lr > 0))
    return set_error(RAFIKI_ERR_INVALID, "need requests, episodes >= 1, gamma in [0, 1] and lr > 0");
  const int64_t cap = n;   // every decision serves at least one request
  std::vector<int32_t> acts(cap);
  std::vector<double> rew(cap), states((size_t)cap * h->D), ret(cap), g(h->lay.n);
  const double scale = 1.0 / (double)h->B.back();
  for (int e = 0; e < episodes; ++e) {
    int64_t steps = 0;
    int rc = rafiki_rl_run_episode(h, arrival_us, n, 1, nullptr, 0, seed + (uint64_t)e, acts.data(), rew.data(),
                                   states.data(), nullptr, cap, &steps, nullptr);
    if (rc) return rc;
    double acc = 0, total = 0;
    for (int64_t t = steps - 1; t >= 0; --t) {
      acc = rew[t] * scale + gamma * acc;
      ret[t] = acc;
      total += rew[t];
    }
    if (out_episode_reward) out_episode_reward[e] = total;
    rc = rafiki_rl_gradient(h, states.data(), acts.data(), ret.data(), steps, c_v, c_e, g.data());
    if (!rc) rc = rafiki_rl_adam_step(h, g.data(), lr);
    if (rc) return rc;
  }
  return RAFIKI_OK;
}

}  // extern "C"

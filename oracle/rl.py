"""Oracle of the RL scheduler's deterministic parts (Section 5.2, multiple models).

TEST INFRASTRUCTURE ONLY (see the package header).

The scheduler picks, for the oldest queued requests, a batch size b from B and a
non-empty model subset v (action space of (2^|M| - 1) * |B| actions).  Its state is
the waiting times of the queued requests (padded with zeros or truncated to a fixed
length) followed by the model status: c(m, b) for every model and candidate size,
and each model's time left on the work already dispatched to it.  A batch's reward
is a(M[v]) * (b - beta * |{s in batch : l(s) > tau}|) (Equation multi_acc_reward),
a(M[v]) the (surrogate) accuracy of the selected ensemble.

Environment reading (the paper describes it in words only):
* each model is an independent server (one model per node or GPU); a batch sent to v
  starts on model m when m is free, occupies it for c(m, b), and completes when the
  last of its models finishes; its requests' latency is completion minus arrival;
* a decision is taken whenever the queue is non-empty and at least one model is free;
  otherwise time advances to the next arrival or to the next model becoming free;
* the batch is the oldest min(b, queue length) requests and costs c(m, b);
* times are integer microseconds; state features are divided by tau.

Policy / value network (actor-critic): two tanh hidden layers shared by a softmax
policy head and a linear value head.  The loss over T transitions (s_t, a_t, R_t) is
  (1/T) sum_t [ -log pi(a_t|s_t) * A_t + c_v (V(s_t) - R_t)^2 - c_e H(pi(.|s_t)) ],
A_t = R_t - V(s_t) held constant, R_t the discounted return.  Parameters update with
Adam.  Everything here is float64.
"""
from itertools import product
from typing import Dict, List, Sequence, Tuple

import numpy as np


# ---------------------------------------------------------------- actions
def actions(n_models: int, B: Sequence[int]) -> List[Tuple[int, int]]:
    """Action index -> (mask, b): masks 1 .. 2^M - 1 outer, batch sizes inner."""
    return [(mask, b) for mask, b in product(range(1, 1 << n_models), B)]


# ---------------------------------------------------------------- environment
class Env:
    def __init__(self, arrivals, B, cost, acc, tau, beta, qlen_feat):
        """cost[m][j] = c(m, B[j]) (us); acc[mask] = a(M[v]) for mask 1 .. 2^M - 1."""
        self.a = [int(x) for x in arrivals]
        self.B = list(B)
        self.cost = [list(map(int, c)) for c in cost]
        self.acc = list(acc)
        self.tau, self.beta, self.L = int(tau), float(beta), int(qlen_feat)
        self.M = len(cost)
        self.acts = actions(self.M, self.B)
        self.t = self.a[0] if self.a else 0
        self.head = 0
        self.arrived = 0
        self.busy = [0] * self.M
        self.lat = [-1] * len(self.a)
        self._advance()

    def done(self) -> bool:
        return self.head >= len(self.a)

    def _advance(self):
        """Move time to the next decision instant (queue non-empty and a model free)."""
        n = len(self.a)
        while self.head < n:
            while self.arrived < n and self.a[self.arrived] <= self.t:
                self.arrived += 1
            free = min(self.busy)
            if self.arrived == self.head:
                self.t = max(self.a[self.arrived], self.t)
                continue
            if free > self.t:
                self.t = free
                continue
            return

    def state(self) -> np.ndarray:
        waits = [(self.t - self.a[i]) / self.tau for i in range(self.head, min(self.arrived, self.head + self.L))]
        waits += [0.0] * (self.L - len(waits))
        costs = [c / self.tau for row in self.cost for c in row]
        left = [max(b - self.t, 0) / self.tau for b in self.busy]
        return np.array(waits + costs + left, dtype=np.float64)

    def step(self, action: int) -> float:
        """Dispatch the action's batch at the current instant; returns its reward."""
        mask, b = self.acts[action]
        j = self.B.index(b)
        nb = min(b, self.arrived - self.head)
        end = 0
        for m in range(self.M):
            if (mask >> m) & 1:
                e = max(self.t, self.busy[m]) + self.cost[m][j]
                self.busy[m] = e
                end = max(end, e)
        over = 0
        for i in range(self.head, self.head + nb):
            self.lat[i] = end - self.a[i]
            over += self.lat[i] > self.tau
        self.head += nb
        self._advance()
        return self.acc[mask] * (nb - self.beta * over)


# ---------------------------------------------------------------- sampling
class SplitMix64:
    """splitmix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
    generators", 2014): the state advances by the golden-ratio increment 0x9E3779B97F4A7C15
    and each output is the state passed through two xor-shift-multiply rounds and a final
    xor-shift; uniform doubles in [0, 1) take the top 53 bits."""
    M64 = (1 << 64) - 1

    def __init__(self, seed: int):
        self.x = seed & self.M64

    def next(self) -> int:
        self.x = (self.x + 0x9E3779B97F4A7C15) & self.M64
        z = self.x
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & self.M64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & self.M64
        return z ^ (z >> 31)

    def uniform(self) -> float:
        return (self.next() >> 11) * (1.0 / 9007199254740992.0)


def sample_action(pi: Sequence[float], u: float) -> int:
    """Inverse-CDF draw: the first action whose running sum of probabilities (in action
    order) exceeds u; the last action if rounding leaves the sum at or below u."""
    c = 0.0
    for i, p in enumerate(pi):
        c += float(p)
        if u < c:
            return i
    return len(pi) - 1


def argmax_action(pi: Sequence[float]) -> int:
    """The most probable action, lowest index on ties."""
    return int(np.argmax(np.asarray(pi)))


# ---------------------------------------------------------------- network
def param_shapes(D: int, H: int, A: int):
    return [("W1", (H, D)), ("b1", (H,)), ("W2", (H, H)), ("b2", (H,)), ("Wp", (A, H)), ("bp", (A,)),
            ("Wv", (1, H)), ("bv", (1,))]


def unflatten(theta: np.ndarray, D: int, H: int, A: int) -> Dict[str, np.ndarray]:
    out, k = {}, 0
    for name, shp in param_shapes(D, H, A):
        size = int(np.prod(shp))
        out[name] = theta[k:k + size].reshape(shp)
        k += size
    assert k == theta.size
    return out


def forward(theta, s, D, H, A):
    """Policy probabilities [A] and value for one state."""
    p = unflatten(theta, D, H, A)
    h1 = np.tanh(p["W1"] @ s + p["b1"])
    h2 = np.tanh(p["W2"] @ h1 + p["b2"])
    z = p["Wp"] @ h2 + p["bp"]
    z = z - z.max()
    pi = np.exp(z) / np.exp(z).sum()
    v = float((p["Wv"] @ h2 + p["bv"])[0])
    return pi, v


def loss(theta, S, acts_taken, R, D, H, A, c_v, c_e, adv=None):
    """The actor-critic loss above.  `adv` (per transition) defaults to R - V(s) under
    theta; pass it explicitly to hold it constant (its gradient is not taken)."""
    T = len(R)
    tot = 0.0
    for i, (s, a, r) in enumerate(zip(S, acts_taken, R)):
        pi, v = forward(theta, s, D, H, A)
        adv_i = r - v if adv is None else adv[i]
        ent = -float(np.sum(pi * np.log(pi)))
        tot += -np.log(pi[a]) * adv_i + c_v * (v - r) ** 2 - c_e * ent
    return tot / T


def grad(theta, S, acts_taken, R, D, H, A, c_v, c_e):
    """Gradient of loss() by backpropagation, the advantage held constant."""
    p = unflatten(theta, D, H, A)
    g = {k: np.zeros_like(v) for k, v in p.items()}
    T = len(R)
    for s, a, r in zip(S, acts_taken, R):
        h1 = np.tanh(p["W1"] @ s + p["b1"])
        h2 = np.tanh(p["W2"] @ h1 + p["b2"])
        z = p["Wp"] @ h2 + p["bp"]
        z = z - z.max()
        pi = np.exp(z) / np.exp(z).sum()
        v = float((p["Wv"] @ h2 + p["bv"])[0])
        adv = r - v
        logpi = np.log(pi)
        ent = -float(np.sum(pi * logpi))
        # d/dz of -log pi_a * adv: (pi - onehot) * adv
        dz = pi.copy()
        dz[a] -= 1.0
        dz *= adv
        # d/dz of -c_e * H: c_e * pi * (log pi + H)
        dz += c_e * pi * (logpi + ent)
        dv = 2.0 * c_v * (v - r)
        g["Wp"] += np.outer(dz, h2)
        g["bp"] += dz
        g["Wv"] += dv * h2[None, :]
        g["bv"] += dv
        dh2 = p["Wp"].T @ dz + dv * p["Wv"][0]
        da2 = dh2 * (1.0 - h2 * h2)
        g["W2"] += np.outer(da2, h1)
        g["b2"] += da2
        dh1 = p["W2"].T @ da2
        da1 = dh1 * (1.0 - h1 * h1)
        g["W1"] += np.outer(da1, s)
        g["b1"] += da1
    return np.concatenate([g[name].ravel() for name, _ in param_shapes(D, H, A)]) / T


def adam_step(theta, m, v, g, step, lr, b1=0.9, b2=0.999, eps=1e-8):
    """One Adam update (Kingma and Ba), bias-corrected; returns new (theta, m, v)."""
    m = b1 * m + (1 - b1) * g
    v = b2 * v + (1 - b2) * g * g
    mh = m / (1 - b1 ** step)
    vh = v / (1 - b2 ** step)
    return theta - lr * mh / (np.sqrt(vh) + eps), m, v


def discounted_returns(rewards: Sequence[float], gamma: float) -> np.ndarray:
    out = np.zeros(len(rewards))
    acc = 0.0
    for i in range(len(rewards) - 1, -1, -1):
        acc = rewards[i] + gamma * acc
        out[i] = acc
    return out

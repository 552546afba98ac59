"""Pins of the RL scheduler oracle (Section 5.2): a hand-worked environment episode,
finite differences for the actor-critic gradient, the closed form of a first Adam step
and of discounted returns, and the size of the action space."""
import json
import os

import numpy as np
import pytest

from oracle import rl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_action_space():
    acts = rl.actions(3, [16, 32, 48, 64])
    assert len(acts) == (2 ** 3 - 1) * 4 and len(set(acts)) == len(acts)
    assert all(m != 0 for m, _ in acts)


def test_env_golden_episode():
    g = json.load(open(os.path.join(GOLDEN, "rl_env_small.json")))
    env = rl.Env(g["arrivals"], g["B"], g["cost"], g["acc"], g["tau"], g["beta"], g["qlen_feat"])
    assert [list(x) for x in env.acts] == g["actions_order"]
    rewards = []
    for k, a in enumerate(g["taken"]):
        assert env.t == g["expected_times"][k]
        assert np.allclose(env.state(), g["expected_states"][k], atol=1e-15)
        rewards.append(env.step(a))
    assert env.done()
    assert rewards == pytest.approx(g["expected_rewards"], abs=1e-15)
    assert env.lat == g["expected_latency"]


def test_gradient_matches_finite_differences():
    rng = np.random.default_rng(0)
    D, H, A = 7, 5, 4
    n = sum(int(np.prod(s)) for _, s in rl.param_shapes(D, H, A))
    theta = rng.standard_normal(n) * 0.5
    S = rng.standard_normal((6, D))
    acts = rng.integers(0, A, 6)
    R = rng.standard_normal(6)
    c_v, c_e = 0.5, 0.03
    adv = np.array([r - rl.forward(theta, s, D, H, A)[1] for s, r in zip(S, R)])
    g = rl.grad(theta, S, acts, R, D, H, A, c_v, c_e)
    eps = 1e-6
    fd = np.zeros(n)
    for i in range(n):
        e = np.zeros(n)
        e[i] = eps
        fd[i] = (rl.loss(theta + e, S, acts, R, D, H, A, c_v, c_e, adv) -
                 rl.loss(theta - e, S, acts, R, D, H, A, c_v, c_e, adv)) / (2 * eps)
    assert np.abs(g - fd).max() <= 1e-7 * max(1.0, np.abs(fd).max())


def test_forward_is_a_distribution_and_softmax_shift_invariant():
    rng = np.random.default_rng(1)
    D, H, A = 5, 4, 6
    n = sum(int(np.prod(s)) for _, s in rl.param_shapes(D, H, A))
    theta = rng.standard_normal(n)
    s = rng.standard_normal(D)
    pi, v = rl.forward(theta, s, D, H, A)
    assert pi.sum() == pytest.approx(1.0, abs=1e-15) and (pi > 0).all()
    p = rl.unflatten(theta.copy(), D, H, A)
    t2 = theta.copy()
    rl.unflatten(t2, D, H, A)["bp"][:] += 3.0          # adding a constant to every logit
    pi2, v2 = rl.forward(t2, s, D, H, A)
    assert np.allclose(pi, pi2, atol=1e-14) and v == v2


def test_first_adam_step_closed_form():
    """With zero moments, the first bias-corrected step is lr * g / (|g| + eps)."""
    g = np.array([0.5, -2.0, 1e-3, 0.0])
    th, m, v = rl.adam_step(np.zeros(4), np.zeros(4), np.zeros(4), g, 1, lr=0.01)
    assert np.allclose(th, -0.01 * g / (np.abs(g) + 1e-8), atol=1e-15)


def test_discounted_returns():
    assert np.allclose(rl.discounted_returns([1.0] * 5, 0.5), [(1 - 0.5 ** k) / 0.5 for k in range(5, 0, -1)])
    assert rl.discounted_returns([2.0, 0.0, 1.0], 0.9).tolist() == pytest.approx([2.0 + 0.81, 0.9, 1.0])


def test_splitmix64_reference_sequence():
    """The generator's published reference outputs for seed 0 (the sequence used to
    seed the xorshift/xoroshiro family), and uniforms in [0, 1) from the top 53 bits."""
    g = rl.SplitMix64(0)
    assert [g.next() for _ in range(4)] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F,
                                            0xF88BB8A8724C81EC]
    g = rl.SplitMix64(0)
    assert g.uniform() == (0xE220A8397B1DCDAF >> 11) / 2.0 ** 53


def test_action_selection():
    pi = [0.1, 0.2, 0.3, 0.4]
    assert [rl.sample_action(pi, u) for u in (0.0, 0.099, 0.1, 0.35, 0.61, 0.999)] == [0, 0, 1, 2, 3, 3]
    assert rl.sample_action([0.5, 0.5 - 1e-17], 1.0 - 1e-17) == 1       # rounding leaves the sum short: last
    assert rl.argmax_action([0.2, 0.4, 0.4]) == 1                      # ties: lowest index

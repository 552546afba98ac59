"""Seeded request-arrival process of the serving experiments (Section 7.2).

The arrival rate follows a sine over a cycle of period T,
    r(t) = gamma * sin(2 pi t / T) + r0,
scaled to a reference throughput r_ref (the slowest or the summed throughput of the
models): the rate exceeds r_ref during 20% of each cycle, centred on the peak, and the
peak is 1.1 r_ref (Equations (r1) and (r2), read with the phase 2 pi t / T).  A simulator
invoked every `step_us` microseconds adds step * r(t) * (1 + phi) requests, phi drawn
from N(0, 0.1) (standard deviation 0.1); the fractional part carries to the next step so
that the mean rate is kept.  All requests added by one invocation arrive at its time.

Only arrival times are produced here (integer microseconds); the scheduler that serves
them is not part of this package.
"""
import math
from typing import Tuple

import numpy as np


def sine_coefficients(r_ref: float) -> Tuple[float, float]:
    """(gamma, r0) such that r >= r_ref on 20% of the cycle and max r = 1.1 r_ref."""
    s = math.cos(0.2 * math.pi)          # sin(pi/2 - 0.2 pi): edge of the 20% window
    gamma = 0.1 * r_ref / (1.0 - s)
    return gamma, 1.1 * r_ref - gamma


def sine_rate(t_us, r_ref: float, period_us: float):
    gamma, r0 = sine_coefficients(r_ref)
    return gamma * np.sin(2.0 * np.pi * np.asarray(t_us, dtype=np.float64) / period_us) + r0


def sine_arrivals(r_ref: float, period_us: int, duration_us: int, step_us: int, seed: int = 0,
                  noise: float = 0.1) -> np.ndarray:
    """Arrival times (int64 microseconds, non-decreasing) over [0, duration_us)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    times = np.arange(0, duration_us, step_us, dtype=np.int64)
    phi = rng.standard_normal(times.size) * noise
    want = step_us * 1e-6 * sine_rate(times, r_ref, period_us) * (1.0 + phi)
    out = []
    carry = 0.0
    for t, w in zip(times, want):
        carry += max(w, 0.0)
        k = int(math.floor(carry))
        carry -= k
        out.extend([int(t)] * k)
    return np.asarray(out, dtype=np.int64)

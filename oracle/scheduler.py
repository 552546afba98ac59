"""Oracle of the greedy batch-size scheduler (Section 5.1, Algorithm "Inference").

TEST INFRASTRUCTURE ONLY (see the package header).

One model serves a FIFO queue one batch at a time.  Whenever the model is free, the
policy looks at the queue:
* with at least max(B) requests queued, the oldest max(B) are served at once;
* otherwise b is the largest candidate size not above the queue length, and the oldest
  b are served as soon as c(b) + w(q_0) + delta >= tau, w(q_0) being the waiting time
  of the oldest queued request; with no such b (fewer requests than min(B)) it waits.

Time is kept in integer microseconds, so every comparison is exact.  A batch started
at time t finishes at t + c(b); its requests' latency l(s) is that finish time minus
their arrival time.  The objective of Equation (single) is the mean exceeding time
sum(max(0, l(s) - tau)) / |S|.
"""
from typing import Dict, List, Sequence, Tuple

import numpy as np


def greedy_decide(B: Sequence[int], cost: Dict[int, int], queue_len: int, oldest_wait: int,
                  tau: int, delta: int) -> int:
    """Batch size to serve now, or 0 to keep waiting (Algorithm "Inference")."""
    bmax = max(B)
    if queue_len >= bmax:
        return bmax
    fitting = [b for b in B if b <= queue_len]
    if not fitting:
        return 0
    b = max(fitting)
    if cost[b] + oldest_wait + delta >= tau:
        return b
    return 0


def simulate_greedy(arrivals: Sequence[int], B: Sequence[int], cost: Dict[int, int], tau: int, delta: int):
    """Event-driven run of the policy over requests arriving at the given times
    (non-decreasing, microseconds).  The decision only changes when a request arrives,
    when the model becomes free, or when the oldest request's wait reaches
    tau - delta - c(b); the simulation visits exactly those instants.

    Returns (latency per request, -1 for requests never served, and the list of
    dispatches (start time, batch size, queue length, oldest wait))."""
    a = [int(x) for x in arrivals]
    n = len(a)
    lat = [-1] * n
    disp: List[Tuple[int, int, int, int]] = []
    t = a[0] if n else 0
    head = 0        # oldest request not yet served
    arrived = 0     # requests with arrival time <= t
    while True:
        while arrived < n and a[arrived] <= t:
            arrived += 1
        qlen = arrived - head
        if qlen == 0:
            if arrived == n:
                break
            t = a[arrived]
            continue
        wait = t - a[head]
        b = greedy_decide(B, cost, qlen, wait, tau, delta)
        if b > 0:
            disp.append((t, b, qlen, wait))
            done = t + cost[b]
            for i in range(head, head + b):
                lat[i] = done - a[i]
            head += b
            t = done
            continue
        nxt = a[arrived] if arrived < n else None
        fitting = [x for x in B if x <= qlen]
        if fitting:
            deadline = a[head] + tau - delta - cost[max(fitting)]
            nxt = deadline if nxt is None else min(nxt, deadline)
        if nxt is None:
            break            # fewer than min(B) requests left and none arriving
        t = nxt
    return lat, disp


def serving_stats(latency: Sequence[int], tau: int) -> dict:
    """Equation (single) objective and overdue counts over all requests (a request never
    served counts as unserved, not in the exceeding time)."""
    lat = np.asarray(latency, dtype=np.int64)
    served = lat >= 0
    exceed = np.maximum(lat[served] - tau, 0)
    return {"requests": int(lat.size), "served": int(served.sum()),
            "overdue": int((lat[served] > tau).sum()),
            "mean_exceeding_us": float(exceed.sum() / max(lat.size, 1))}


def simulate_greedy_multi(arrivals: Sequence[int], policies) -> Tuple[List[int], list]:
    """Several independent servers (one model each) sharing the FIFO queue (Section 5.2:
    each model an independent server; Section 5.1: each applies the greedy policy of
    Algorithm "Inference" whenever it is free).  At each instant the free servers are
    visited in index order, and the visit is repeated until none of them dispatches: a
    dispatch changes the queue (its length and its oldest request), and a server that
    declined before it must see the new queue at the same instant.  Each takes a batch
    of the oldest queued requests chosen by its own policy (B, cost dict, tau, delta).

    Returns (latency per request or -1, dispatches (start, batch size, queue length,
    oldest wait, server))."""
    a = [int(x) for x in arrivals]
    n = len(a)
    lat = [-1] * n
    disp = []
    free_at = [None] * len(policies)      # None: never used
    t = a[0] if n else 0
    head = arrived = 0
    while head < n:
        while arrived < n and a[arrived] <= t:
            arrived += 1
        again = True
        while again:
            again = False
            for k, (B, cost, tau, delta) in enumerate(policies):
                if (free_at[k] is not None and free_at[k] > t) or arrived == head:
                    continue
                b = greedy_decide(B, cost, arrived - head, t - a[head], tau, delta)
                if b == 0:
                    continue
                disp.append((t, b, arrived - head, t - a[head], k))
                for i in range(head, head + b):
                    lat[i] = t + cost[b] - a[i]
                head += b
                free_at[k] = t + cost[b]
                again = True
        if head >= n:
            break
        cands = [a[arrived]] if arrived < n else []
        for k, (B, cost, tau, delta) in enumerate(policies):
            if free_at[k] is not None and free_at[k] > t:
                cands.append(free_at[k])
            elif arrived > head:
                fitting = [x for x in B if x <= arrived - head]
                if fitting:
                    cands.append(a[head] + tau - delta - cost[max(fitting)])
        if not cands:
            break
        # every free server declined the final queue at t, so its deadline lies after t
        assert min(cands) > t, (min(cands), t)
        t = min(cands)
    return lat, disp

"""Scalar pure-Python loops for tiny inputs: an independent second reading of the
layer definitions, used only to pin the vectorised oracle.

TEST INFRASTRUCTURE ONLY.  Each function follows the textbook definition directly,
one output element at a time, on nested Python lists or small numpy arrays.
"""
import math


def conv2d(x, w, stride, pad, bias=None):
    """x [N][C][H][W], w [O][C][kh][kw]: cross-correlation with zero padding."""
    N, C, H, W = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    O, kh, kw = len(w), len(w[0][0]), len(w[0][0][0])
    Ho = (H + 2 * pad - kh) // stride + 1
    Wo = (W + 2 * pad - kw) // stride + 1
    out = [[[[0.0] * Wo for _ in range(Ho)] for _ in range(O)] for _ in range(N)]
    for n in range(N):
        for o in range(O):
            for yy in range(Ho):
                for xx in range(Wo):
                    s = 0.0 if bias is None else float(bias[o])
                    for c in range(C):
                        for u in range(kh):
                            for v in range(kw):
                                iy = yy * stride + u - pad
                                ix = xx * stride + v - pad
                                if 0 <= iy < H and 0 <= ix < W:
                                    s += float(w[o][c][u][v]) * float(x[n][c][iy][ix])
                    out[n][o][yy][xx] = s
    return out


def maxpool2d(x, k, stride, pad):
    N, C, H, W = len(x), len(x[0]), len(x[0][0]), len(x[0][0][0])
    Ho = (H + 2 * pad - k) // stride + 1
    Wo = (W + 2 * pad - k) // stride + 1
    out = [[[[0.0] * Wo for _ in range(Ho)] for _ in range(C)] for _ in range(N)]
    for n in range(N):
        for c in range(C):
            for yy in range(Ho):
                for xx in range(Wo):
                    m = -math.inf
                    for u in range(k):
                        for v in range(k):
                            iy, ix = yy * stride + u - pad, xx * stride + v - pad
                            if 0 <= iy < H and 0 <= ix < W:
                                m = max(m, float(x[n][c][iy][ix]))
                    out[n][c][yy][xx] = m
    return out


def fc(x, w, bias=None):
    """x [N][I] (already flat), w [O][I]."""
    out = []
    for row in x:
        out.append([(0.0 if bias is None else float(bias[o])) +
                    sum(float(w[o][i]) * float(row[i]) for i in range(len(row))) for o in range(len(w))])
    return out


def conv1d_maxtime(e, w, bias, apply_relu):
    """e [N][L][D], w [F][D][k] -> [N][F]."""
    N, L, D = len(e), len(e[0]), len(e[0][0])
    F, k = len(w), len(w[0][0])
    out = []
    for n in range(N):
        row = []
        for f in range(F):
            best = -math.inf
            for t in range(L - k + 1):
                s = 0.0 if bias is None else float(bias[f])
                for j in range(k):
                    for d in range(D):
                        s += float(e[n][t + j][d]) * float(w[f][d][j])
                if apply_relu:
                    s = max(s, 0.0)
                best = max(best, s)
            row.append(best)
        out.append(row)
    return out


def softmax_row(z):
    m = max(z)
    ex = [math.exp(v - m) for v in z]
    s = sum(ex)
    return [v / s for v in ex]


def greedy_busy_loop(arrivals, B, cost, tau, delta, t_end):
    """The scheduling loop of Algorithm "Inference" stepped literally, one microsecond
    per iteration, until t_end: while the model is free, test the two conditions on the
    current queue; when busy, let time pass.  Returns (latency per request or -1,
    dispatch list of (start, b))."""
    n = len(arrivals)
    lat = [-1] * n
    disp = []
    head, arrived, busy_until = 0, 0, -1
    for t in range(int(arrivals[0]) if n else 0, int(t_end) + 1):
        while arrived < n and arrivals[arrived] <= t:
            arrived += 1
        if t < busy_until:
            continue
        q = arrived - head
        b = 0
        if q >= max(B):
            b = max(B)
        elif q > 0:
            smaller = [x for x in B if x <= q]
            if smaller and cost[max(smaller)] + (t - arrivals[head]) + delta >= tau:
                b = max(smaller)
        if b:
            disp.append((t, b))
            for i in range(head, head + b):
                lat[i] = t + cost[b] - arrivals[i]
            head += b
            busy_until = t + cost[b]
    return lat, disp


def greedy_multi_busy_loop(arrivals, policies, t_end):
    """Several servers sharing one FIFO queue, stepped literally one microsecond per
    iteration until t_end.  At each microsecond every free server, in index order,
    tests the two conditions of Algorithm "Inference" with its own (B, cost, tau, delta)
    on the current queue, and the round of tests is repeated while any server
    dispatched.  Returns (latency per request or -1, dispatch list of (start, b, server))."""
    n = len(arrivals)
    lat = [-1] * n
    disp = []
    head, arrived = 0, 0
    busy_until = [-1] * len(policies)
    for t in range(int(arrivals[0]) if n else 0, int(t_end) + 1):
        while arrived < n and arrivals[arrived] <= t:
            arrived += 1
        again = True
        while again:
            again = False
            for k, (B, cost, tau, delta) in enumerate(policies):
                if t < busy_until[k]:
                    continue
                q = arrived - head
                b = 0
                if q >= max(B):
                    b = max(B)
                elif q > 0:
                    smaller = [x for x in B if x <= q]
                    if smaller and cost[max(smaller)] + (t - arrivals[head]) + delta >= tau:
                        b = max(smaller)
                if b:
                    disp.append((t, b, k))
                    for i in range(head, head + b):
                        lat[i] = t + cost[b] - arrivals[i]
                    head += b
                    busy_until[k] = t + cost[b]
                    again = True
    return lat, disp

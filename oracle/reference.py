"""fp64 CPU oracle of the ensemble-inference hot path.

TEST INFRASTRUCTURE ONLY: imported by tests, the smoke check and the benchmark's CPU
baseline leg, never by the product path.  It shares no code with the HIP library.

What it computes (the paper's inference service, Section 5 and Section 1):
* each deployed model runs its forward pass over the batch of the oldest requests,
  ``m.infer(q_{0:b})`` (Section 5.1, Algorithm "Inference");
* the models selected by the binary vector v (Table 2; Section 5.2, where v = 0 is
  excluded) are combined by averaging their results (Section 1: products ensemble
  several models and average the results), read here as the mean of the per-model
  softmax probabilities, followed by the first-index argmax.

The paper defines no network and no numerics, so each layer below is the textbook
definition, written out in fp64 in NCHW layout:
* conv2d: cross-correlation with zero padding, output size floor((H + 2P - k)/S) + 1;
* inference batch-norm, unfolded: gamma * (x - mean) / sqrt(var + eps) + beta;
* residual add before the ReLU; ReLU = max(0, x);
* max-pool with -inf padding; global average pool = sum / (H * W);
* FC: W x + b, a spatial input flattened in (c, h, w) order;
* TextCNN front: embedding gather, valid conv1d + bias + ReLU, max over time,
  concatenation in layer order;
* softmax with the max subtracted; ensemble mean; argmax = lowest index among the maxima.

``act="bf16"`` rounds every tensor a model stores between layers (all layer outputs
except the final logits) to the nearest bfloat16, ties to even: the storage
precision of the bf16 workloads.  ``act=None`` keeps fp64 throughout.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# Operation codes of the layer lists (plain integers; see the workload package).
_CONV2D, _MAXPOOL2D, _GAP, _FC, _EMBEDDING, _CONV1D_MAXTIME, _CONCAT = 1, 2, 3, 4, 5, 6, 7


def to_bf16_rne(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value of each fp64 element (8 significant bits, ties to even).

    x = m * 2**e with 0.5 <= |m| < 1 (frexp); m * 2**8 is rounded half-to-even with
    rint, which keeps 8 significant bits.  Normal-range finite inputs only.
    """
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def conv2d(x: np.ndarray, w: np.ndarray, stride: int = 1, pad: int = 0,
           bias: Optional[np.ndarray] = None) -> np.ndarray:
    """out[n, o, y, x] = sum_{c, u, v} w[o, c, u, v] * xpad[n, c, y*S + u, x*S + v] (+ bias[o]).

    x: [N, C, H, W]; w: [O, C, kh, kw]; zero padding of width ``pad`` on each side.
    Written as a sum over the kernel taps (u, v) of channel contractions.
    """
    x = np.asarray(x, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, c, h, wd = x.shape
    o, c2, kh, kw = w.shape
    assert c == c2, (c, c2)
    ho = (h + 2 * pad - kh) // stride + 1
    wo = (wd + 2 * pad - kw) // stride + 1
    # channel-major padded copy [C, N, H + 2P, W + 2P]: each tap is one 2-D product
    xp = np.zeros((c, n, h + 2 * pad, wd + 2 * pad), dtype=np.float64)
    xp[:, :, pad:pad + h, pad:pad + wd] = x.transpose(1, 0, 2, 3)
    acc = np.zeros((o, n * ho * wo), dtype=np.float64)
    for u in range(kh):
        for v in range(kw):
            patch = xp[:, :, u:u + stride * (ho - 1) + 1:stride, v:v + stride * (wo - 1) + 1:stride]
            acc += np.ascontiguousarray(w[:, :, u, v]) @ patch.reshape(c, n * ho * wo)
    out = np.ascontiguousarray(acc.reshape(o, n, ho, wo).transpose(1, 0, 2, 3))
    if bias is not None:
        out += np.asarray(bias, dtype=np.float64)[None, :, None, None]
    return out


def batchnorm(x: np.ndarray, gamma, beta, mean, var, eps: float) -> np.ndarray:
    """Inference batch-norm over the channel axis 1: gamma * (x - mean) / sqrt(var + eps) + beta."""
    shp = (1, -1) + (1,) * (x.ndim - 2)
    g = np.asarray(gamma, np.float64).reshape(shp)
    b = np.asarray(beta, np.float64).reshape(shp)
    mu = np.asarray(mean, np.float64).reshape(shp)
    va = np.asarray(var, np.float64).reshape(shp)
    return g * (x - mu) / np.sqrt(va + eps) + b


def relu(x: np.ndarray) -> np.ndarray:
    return np.maximum(x, 0.0)


def maxpool2d(x: np.ndarray, k: int, stride: int, pad: int) -> np.ndarray:
    """Max over each k x k window (stride S, padding P filled with -inf).  x: [N, C, H, W]."""
    n, c, h, wd = x.shape
    ho = (h + 2 * pad - k) // stride + 1
    wo = (wd + 2 * pad - k) // stride + 1
    xp = np.full((n, c, h + 2 * pad, wd + 2 * pad), -np.inf, dtype=np.float64)
    xp[:, :, pad:pad + h, pad:pad + wd] = x
    out = np.full((n, c, ho, wo), -np.inf, dtype=np.float64)
    for u in range(k):
        for v in range(k):
            out = np.maximum(out, xp[:, :, u:u + stride * (ho - 1) + 1:stride, v:v + stride * (wo - 1) + 1:stride])
    return out


def global_avgpool(x: np.ndarray) -> np.ndarray:
    """[N, C, H, W] -> [N, C]: sum over the H*W positions divided by H*W."""
    n, c, h, wd = x.shape
    return x.reshape(n, c, h * wd).sum(axis=2) / float(h * wd)


def fc(x: np.ndarray, w: np.ndarray, bias: Optional[np.ndarray] = None) -> np.ndarray:
    """z[n, o] = sum_i w[o, i] * flat(x)[n, i] (+ bias[o]); flat() is row-major, i.e. (c, h, w)."""
    x = np.asarray(x, dtype=np.float64).reshape(x.shape[0], -1)
    z = x @ np.asarray(w, dtype=np.float64).T
    if bias is not None:
        z = z + np.asarray(bias, dtype=np.float64)[None, :]
    return z


def embedding(tokens: np.ndarray, table: np.ndarray) -> np.ndarray:
    """[N, L] int ids -> [N, L, D] rows of the table."""
    return np.asarray(table, dtype=np.float64)[np.asarray(tokens, dtype=np.int64)]


def conv1d_maxtime(e: np.ndarray, w: np.ndarray, bias: Optional[np.ndarray], apply_relu: bool) -> np.ndarray:
    """Valid conv1d over time, bias, ReLU, then max over time.

    e: [N, L, D]; w: [F, D, k].  y[n, f, t] = sum_{j<k} sum_d e[n, t + j, d] * w[f, d, j] (+ bias[f]),
    t = 0 .. L - k; the result is max_t of (ReLU of) y, shape [N, F].
    """
    e = np.asarray(e, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    n, L, d = e.shape
    f, d2, k = w.shape
    assert d == d2
    T = L - k + 1
    y = np.zeros((n * T, f), dtype=np.float64)
    for j in range(k):
        y += e[:, j:j + T, :].reshape(n * T, d) @ np.ascontiguousarray(w[:, :, j].T)
    y = y.reshape(n, T, f)
    if bias is not None:
        y += np.asarray(bias, dtype=np.float64)[None, None, :]
    if apply_relu:
        y = relu(y)
    return y.max(axis=1)


def concat(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Join along the channel axis 1, ``a`` first."""
    return np.concatenate([a, b], axis=1)


def softmax(z: np.ndarray) -> np.ndarray:
    """Row softmax: exp(z - max z) / sum exp(z - max z)."""
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def combine_mean(probs: Sequence[np.ndarray]) -> np.ndarray:
    """Mean over the selected models of their [N, C] probability rows."""
    return sum(np.asarray(p, dtype=np.float64) for p in probs) / float(len(probs))


def argmax_first(p: np.ndarray) -> np.ndarray:
    """Per row, the lowest class index among those attaining the maximum."""
    return np.argmax(p, axis=-1).astype(np.int32)


def _layer_forward(L, P, tensors: Dict[int, np.ndarray], batch) -> np.ndarray:
    src = batch if L.input == -1 else tensors[L.input]
    op = L.op
    if op == _CONV2D:
        y = conv2d(src, P.weight, L.stride, L.pad, P.bias if L.bias else None)
        if L.bn:
            y = batchnorm(y, P.bn_gamma, P.bn_beta, P.bn_mean, P.bn_var, P.bn_eps)
        if L.input2 >= 0:
            y = y + tensors[L.input2]
        return relu(y) if L.relu else y
    if op == _MAXPOOL2D:
        assert L.kh == L.kw
        return maxpool2d(src, L.kh, L.stride, L.pad)
    if op == _GAP:
        return global_avgpool(src)
    if op == _FC:
        y = fc(src, P.weight, P.bias if L.bias else None)
        return relu(y) if L.relu else y
    if op == _EMBEDDING:
        return embedding(src, P.weight)
    if op == _CONV1D_MAXTIME:
        return conv1d_maxtime(src, P.weight, P.bias if L.bias else None, L.relu)
    if op == _CONCAT:
        return concat(src, tensors[L.input2])
    raise ValueError(f"unknown op {op}")


def run_model(spec, params, batch: np.ndarray, act: Optional[str] = None,
              chunk: int = 8) -> np.ndarray:
    """Logits [N, n_classes] of one model over a request batch.

    ``batch`` is NCHW images or [N, L] token ids.  Images are independent, so the
    batch is processed ``chunk`` requests at a time (no effect on the result).
    """
    n = batch.shape[0]
    outs = []
    for s in range(0, n, chunk):
        b = batch[s:s + chunk]
        if b.dtype.kind == "f":
            b = b.astype(np.float64)
        tensors: Dict[int, np.ndarray] = {}
        last = len(spec.layers) - 1
        for i, (L, P) in enumerate(zip(spec.layers, params.layers)):
            y = _layer_forward(L, P, tensors, b)
            if act == "bf16" and i != last:
                y = to_bf16_rne(y)
            elif act not in (None, "bf16"):
                raise ValueError(act)
            tensors[i] = y
        outs.append(tensors[last])
    return np.concatenate(outs, axis=0)


def ensemble(specs, params, batch: np.ndarray, mask: int, act: Optional[str] = None,
             logits: Optional[List[np.ndarray]] = None):
    """Ensemble result over the models whose bit is set in ``mask`` (bit m = model m).

    Returns (probs [N, C], labels [N], per-model logits list aligned with ``specs``,
    entries None for unselected models).  ``logits`` may pass precomputed per-model
    logits (as returned before) to avoid recomputation.
    """
    if mask == 0:
        raise ValueError("the selection vector must not be all zeros")
    if mask >> len(specs):
        raise ValueError("mask selects a model that does not exist")
    zs: List[Optional[np.ndarray]] = [None] * len(specs)
    probs = []
    for m in range(len(specs)):
        if not (mask >> m) & 1:
            continue
        z = logits[m] if logits is not None and logits[m] is not None else run_model(specs[m], params[m], batch, act)
        zs[m] = z
        probs.append(softmax(z))
    p = combine_mean(probs)
    return p, argmax_first(p), zs


def combine_vote(logits: Sequence[np.ndarray]):
    """Majority vote of the selected models (Section 5.2, the ensemble experiment).

    ``logits`` lists the selected models in priority order (first = highest).  Each
    model votes for its own first-index argmax; the winning class has the most votes,
    and a tie between classes goes to the one predicted by the highest-priority model
    among those tied.  Returns (vote fractions [N, C], labels [N])."""
    preds = [argmax_first(np.asarray(z, dtype=np.float64)) for z in logits]
    n, c = np.asarray(logits[0]).shape
    votes = np.zeros((n, c), dtype=np.float64)
    for pr in preds:
        votes[np.arange(n), pr] += 1.0
    labels = np.zeros(n, dtype=np.int32)
    for i in range(n):
        best = votes[i].max()
        for pr in preds:                      # priority order
            if votes[i, pr[i]] == best:
                labels[i] = pr[i]
                break
    return votes / float(len(logits)), labels


def ensemble_vote(specs, params, batch: np.ndarray, mask: int, act: Optional[str] = None,
                  logits: Optional[List[np.ndarray]] = None):
    """Majority-vote ensemble over the models selected by ``mask``; model order is the
    priority order.  Returns (vote fractions, labels, per-model logits)."""
    if mask == 0:
        raise ValueError("the selection vector must not be all zeros")
    if mask >> len(specs):
        raise ValueError("mask selects a model that does not exist")
    zs: List[Optional[np.ndarray]] = [None] * len(specs)
    sel = []
    for m in range(len(specs)):
        if not (mask >> m) & 1:
            continue
        z = logits[m] if logits is not None and logits[m] is not None else run_model(specs[m], params[m], batch, act)
        zs[m] = z
        sel.append(z)
    v, lab = combine_vote(sel)
    return v, lab, zs


def model_macs(spec) -> int:
    """Algorithmic multiply-accumulates per request of one model (no padding counted)."""
    shapes: Dict[int, Tuple[int, ...]] = {}
    inp = spec.input_shape
    macs = 0
    for i, L in enumerate(spec.layers):
        src = inp if L.input == -1 else shapes[L.input]
        if L.op == _CONV2D:
            c, h, w = src
            ho = (h + 2 * L.pad - L.kh) // L.stride + 1
            wo = (w + 2 * L.pad - L.kw) // L.stride + 1
            macs += ho * wo * L.c_out * L.c_in * L.kh * L.kw
            shapes[i] = (L.c_out, ho, wo)
        elif L.op == _MAXPOOL2D:
            c, h, w = src
            shapes[i] = (c, (h + 2 * L.pad - L.kh) // L.stride + 1, (w + 2 * L.pad - L.kw) // L.stride + 1)
        elif L.op == _GAP:
            shapes[i] = (src[0],)
        elif L.op == _FC:
            macs += L.c_in * L.c_out
            shapes[i] = (L.c_out,)
        elif L.op == _EMBEDDING:
            shapes[i] = (src[0], L.c_out)
        elif L.op == _CONV1D_MAXTIME:
            T = src[0] - L.kw + 1
            macs += T * L.c_out * L.c_in * L.kw
            shapes[i] = (L.c_out,)
        elif L.op == _CONCAT:
            shapes[i] = (shapes[L.input][0] + shapes[L.input2][0],)
    return macs

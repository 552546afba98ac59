"""ctypes binding of the C ABI in ``include/rafiki_ensemble.h``.

Argument marshalling only: layer lists become ``rafiki_layer`` arrays, torch CUDA
tensors become device pointers, and the current torch stream becomes the
``hipStream_t``.  Every step of the computation runs in the HIP library; if the
library is missing the binding raises instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import List, Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# RAFIKI_LIBRARY names another build of the same sources (the host-sanitizer build)
LIB_PATH = os.environ.get("RAFIKI_LIBRARY") or os.path.join(_PKG, "librafiki_ensemble.so")

RAFIKI_OK, RAFIKI_ERR_INVALID, RAFIKI_ERR_UNSUPPORTED, RAFIKI_ERR_NOMEM, RAFIKI_ERR_HIP = 0, -1, -2, -3, -4
# force_tile: the direct conv kernel wherever it applies (RAFIKI_TILE_DIRECT in the header)
RAFIKI_TILE_DIRECT = 1000
RAFIKI_FP32, RAFIKI_BF16 = 0, 1
RAFIKI_INPUT_IMAGE_NCHW_F32, RAFIKI_INPUT_TOKENS_I32 = 0, 1
EXPORTED = ("rafiki_ensemble_create", "rafiki_ensemble_infer", "rafiki_ensemble_infer_vote",
            "rafiki_ensemble_infer_noalloc", "rafiki_ensemble_model_logits",
            "rafiki_ensemble_info", "rafiki_ensemble_trace", "rafiki_ensemble_trace_read",
            "rafiki_tile_config", "rafiki_ensemble_force_tile", "rafiki_ensemble_get_schedule",
            "rafiki_ensemble_set_schedule", "rafiki_ensemble_get_schedule_pair", "rafiki_ensemble_set_schedule_pair",
            "rafiki_ensemble_get_schedule_tiles", "rafiki_ensemble_set_schedule_tiles",
            "rafiki_ensemble_pairing", "rafiki_ensemble_use_graphs",
            "rafiki_ensemble_graph_stats", "rafiki_combine_mean", "rafiki_combine_vote",
            "rafiki_maxpool_nhwc_bf16", "rafiki_global_avgpool_nhwc_bf16", "rafiki_probe_mfma_bf16",
            "rafiki_probe_hbm_read", "rafiki_probe_mainloop",
            "rafiki_ensemble_destroy", "rafiki_greedy_decide", "rafiki_greedy_simulate", "rafiki_greedy_simulate_multi",
            "rafiki_ensemble_profile", "rafiki_ensemble_serve_greedy", "rafiki_ensemble_serve_greedy_async",
            "rafiki_ensemble_serve_rl",
            "rafiki_rl_create", "rafiki_rl_destroy", "rafiki_rl_info", "rafiki_rl_get_params", "rafiki_rl_set_params",
            "rafiki_rl_forward", "rafiki_rl_gradient", "rafiki_rl_adam_step", "rafiki_rl_run_episode",
            "rafiki_rl_train", "rafiki_last_error")
KERNEL_CLASSES = ("conv_mfma", "splitk_reduce", "conv_f32", "stage", "pool", "embed", "concat", "combine", "vote",
                  "fused_net")

_fp = C.POINTER(C.c_float)


class RafikiGreedyPolicy(C.Structure):
    _fields_ = [("batch_sizes", C.POINTER(C.c_int32)), ("cost_us", C.POINTER(C.c_int64)), ("n_sizes", C.c_int),
                ("tau_us", C.c_int64), ("delta_us", C.c_int64)]


class RafikiDispatch(C.Structure):
    _fields_ = [("start_us", C.c_int64), ("end_us", C.c_int64), ("first", C.c_int64), ("queue_len", C.c_int64),
                ("oldest_wait_us", C.c_int64), ("b", C.c_int32), ("model", C.c_int32)]


class RafikiRLConfig(C.Structure):
    _fields_ = [("n_models", C.c_int), ("batch_sizes", C.POINTER(C.c_int32)), ("n_sizes", C.c_int),
                ("cost_us", C.POINTER(C.c_int64)), ("accuracy", C.POINTER(C.c_double)), ("tau_us", C.c_int64),
                ("beta", C.c_double), ("queue_features", C.c_int), ("hidden", C.c_int)]


DISPATCH_FIELDS = ("start_us", "end_us", "first", "queue_len", "oldest_wait_us", "b", "model")


class RafikiLayer(C.Structure):
    _fields_ = [("op", C.c_int), ("input", C.c_int), ("input2", C.c_int), ("c_in", C.c_int), ("c_out", C.c_int),
                ("kh", C.c_int), ("kw", C.c_int), ("stride", C.c_int), ("pad", C.c_int), ("relu", C.c_int),
                ("weight", _fp), ("bias", _fp), ("bn_gamma", _fp), ("bn_beta", _fp), ("bn_mean", _fp),
                ("bn_var", _fp), ("bn_eps", C.c_float)]


class RafikiModelDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("layers", C.POINTER(RafikiLayer)), ("n_classes", C.c_int)]


class RafikiOpts(C.Structure):
    _fields_ = [("input_kind", C.c_int), ("c", C.c_int), ("h", C.c_int), ("w", C.c_int), ("vocab", C.c_int),
                ("precision", C.c_int), ("max_batch", C.c_int)]


class RafikiTraceRec(C.Structure):
    _fields_ = [("kind", C.c_int), ("model", C.c_int), ("layer", C.c_int), ("flops", C.c_double),
                ("bytes", C.c_double), ("ms", C.c_float), ("tile_cfg", C.c_int), ("splits", C.c_int)]


class RafikiError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"rafiki error {code}: {msg}")
        self.code = code


_lib = None


def load_library(path: str = LIB_PATH):
    """Load the HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"HIP library not built: {path} (run paper_1804_06087_amd.build)")
    lib = C.CDLL(path)
    lib.rafiki_ensemble_create.argtypes = [C.POINTER(RafikiModelDesc), C.c_int, C.POINTER(RafikiOpts),
                                           C.POINTER(C.c_void_p)]
    lib.rafiki_ensemble_infer.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_uint32, C.c_void_p, C.c_void_p,
                                          C.c_void_p]
    lib.rafiki_ensemble_infer_vote.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_uint32, C.c_void_p,
                                               C.c_void_p, C.c_void_p]
    lib.rafiki_ensemble_infer_noalloc.argtypes = [C.c_void_p, C.c_void_p, C.c_int, C.c_uint32, C.c_void_p,
                                                  C.c_void_p, C.c_void_p]
    lib.rafiki_ensemble_model_logits.argtypes = [C.c_void_p, C.c_int, C.c_void_p, C.c_int, C.c_void_p, C.c_void_p]
    lib.rafiki_ensemble_info.argtypes = [C.c_void_p, C.POINTER(C.c_int), C.POINTER(C.c_int), C.POINTER(C.c_int)]
    lib.rafiki_ensemble_destroy.argtypes = [C.c_void_p]
    lib.rafiki_ensemble_trace.argtypes = [C.c_void_p, C.c_int]
    lib.rafiki_ensemble_trace_read.argtypes = [C.c_void_p, C.POINTER(RafikiTraceRec), C.c_int, C.POINTER(C.c_int)]
    lib.rafiki_tile_config.argtypes = [C.c_int] + [C.POINTER(C.c_int)] * 5
    lib.rafiki_ensemble_force_tile.argtypes = [C.c_void_p, C.c_int]
    lib.rafiki_ensemble_get_schedule.argtypes = [C.c_void_p, C.c_int, C.c_uint32, C.POINTER(C.c_int),
                                                 C.POINTER(C.c_int)]
    lib.rafiki_ensemble_set_schedule.argtypes = [C.c_void_p, C.c_int, C.c_uint32, C.c_int, C.c_int]
    lib.rafiki_ensemble_get_schedule_pair.argtypes = [C.c_void_p, C.c_int, C.c_uint32, C.POINTER(C.c_int),
                                                      C.POINTER(C.c_int)]
    lib.rafiki_ensemble_set_schedule_pair.argtypes = [C.c_void_p, C.c_int, C.c_uint32, C.c_int, C.c_int]
    lib.rafiki_ensemble_get_schedule_tiles.argtypes = [C.c_void_p, C.c_int, C.c_uint32, C.POINTER(C.c_int)]
    lib.rafiki_ensemble_set_schedule_tiles.argtypes = [C.c_void_p, C.c_int, C.c_uint32, C.c_int]
    lib.rafiki_ensemble_pairing.argtypes = [C.c_void_p, C.c_int, C.c_int, C.POINTER(C.c_int)]
    lib.rafiki_ensemble_use_graphs.argtypes = [C.c_void_p, C.c_int]
    lib.rafiki_ensemble_graph_stats.argtypes = [C.c_void_p, C.POINTER(C.c_int), C.POINTER(C.c_longlong),
                                                C.POINTER(C.c_longlong)]
    lib.rafiki_combine_mean.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p]
    lib.rafiki_combine_vote.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_void_p, C.c_void_p]
    lib.rafiki_maxpool_nhwc_bf16.argtypes = [C.c_void_p, C.c_void_p] + [C.c_int] * 7 + [C.c_void_p]
    lib.rafiki_probe_mfma_bf16.argtypes = [C.c_int, C.c_int, C.c_void_p, C.c_void_p]
    lib.rafiki_probe_hbm_read.argtypes = [C.c_void_p, C.c_longlong, C.c_int, C.c_void_p, C.c_void_p]
    lib.rafiki_probe_mainloop.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_void_p]
    lib.rafiki_global_avgpool_nhwc_bf16.argtypes = [C.c_void_p, C.c_void_p] + [C.c_int] * 4 + [C.c_void_p]
    P = C.POINTER
    lib.rafiki_greedy_decide.argtypes = [P(RafikiGreedyPolicy), C.c_int64, C.c_int64, P(C.c_int32)]
    lib.rafiki_greedy_simulate.argtypes = [P(RafikiGreedyPolicy), P(C.c_int64), C.c_int64, P(C.c_int64),
                                           P(RafikiDispatch), C.c_int64, P(C.c_int64)]
    lib.rafiki_greedy_simulate_multi.argtypes = [P(RafikiGreedyPolicy), C.c_int, P(C.c_int64), C.c_int64,
                                                 P(C.c_int64), P(RafikiDispatch), C.c_int64, P(C.c_int64)]
    D = P(C.c_double)
    lib.rafiki_ensemble_serve_rl.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, P(C.c_int64), C.c_int64, C.c_int,
                                             C.c_uint64, C.c_void_p, C.c_void_p, P(C.c_int64),
                                             P(RafikiDispatch), P(C.c_int32), D, C.c_int64, P(C.c_int64),
                                             C.c_void_p]
    lib.rafiki_rl_create.argtypes = [P(RafikiRLConfig), C.c_uint64, P(C.c_void_p)]
    lib.rafiki_rl_destroy.argtypes = [C.c_void_p]
    lib.rafiki_rl_info.argtypes = [C.c_void_p, P(C.c_int), P(C.c_int), P(C.c_int64)]
    lib.rafiki_rl_get_params.argtypes = [C.c_void_p, D, C.c_int64]
    lib.rafiki_rl_set_params.argtypes = [C.c_void_p, D, C.c_int64]
    lib.rafiki_rl_forward.argtypes = [C.c_void_p, D, D, D]
    lib.rafiki_rl_gradient.argtypes = [C.c_void_p, D, P(C.c_int32), D, C.c_int64, C.c_double, C.c_double, D]
    lib.rafiki_rl_adam_step.argtypes = [C.c_void_p, D, C.c_double]
    lib.rafiki_rl_run_episode.argtypes = [C.c_void_p, P(C.c_int64), C.c_int64, C.c_int, P(C.c_int32), C.c_int64,
                                          C.c_uint64, P(C.c_int32), D, D, P(C.c_int64), C.c_int64, P(C.c_int64),
                                          P(C.c_int64)]
    lib.rafiki_rl_train.argtypes = [C.c_void_p, P(C.c_int64), C.c_int64, C.c_int, C.c_double, C.c_double,
                                    C.c_double, C.c_double, C.c_uint64, D]
    lib.rafiki_ensemble_profile.argtypes = [C.c_void_p, C.c_void_p, P(C.c_int32), C.c_int, C.c_uint32, C.c_int,
                                            C.c_void_p, C.c_void_p, P(C.c_int64), C.c_void_p]
    lib.rafiki_ensemble_serve_greedy.argtypes = [C.c_void_p, C.c_void_p, P(C.c_int64), C.c_int64,
                                                 P(RafikiGreedyPolicy), C.c_uint32, C.c_int, C.c_void_p, C.c_void_p,
                                                 P(C.c_int64), P(RafikiDispatch), C.c_int64, P(C.c_int64),
                                                 C.c_void_p]
    lib.rafiki_ensemble_serve_greedy_async.argtypes = [C.c_void_p, C.c_void_p, P(C.c_int64), C.c_int64,
                                                       P(RafikiGreedyPolicy), C.c_uint32, C.c_void_p, C.c_void_p,
                                                       P(C.c_int64), P(RafikiDispatch), C.c_int64, P(C.c_int64),
                                                       C.c_void_p]
    lib.rafiki_last_error.restype = C.c_char_p
    for name in EXPORTED[:-1]:
        getattr(lib, name).restype = C.c_int
    _lib = lib
    return lib


def last_error() -> str:
    return load_library().rafiki_last_error().decode()


def _check(rc: int):
    if rc != RAFIKI_OK:
        raise RafikiError(rc, last_error())


def _fptr(a: Optional[np.ndarray], keep: list):
    if a is None:
        return None
    a = np.ascontiguousarray(a, dtype=np.float32)
    keep.append(a)
    return a.ctypes.data_as(_fp)


def _ptr(t) -> int:
    """Device pointer of a torch tensor (or a raw integer address)."""
    if t is None:
        return 0
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _i32p(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_int32))


def _i64p(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_int64))


def make_policy(batch_sizes, cost_us, tau_us: int, delta_us: int, keep: list) -> RafikiGreedyPolicy:
    B = np.ascontiguousarray(batch_sizes, dtype=np.int32)
    c = np.ascontiguousarray(cost_us, dtype=np.int64)
    keep += [B, c]
    p = RafikiGreedyPolicy()
    p.batch_sizes, p.cost_us, p.n_sizes = _i32p(B), _i64p(c), int(B.size)
    p.tau_us, p.delta_us = int(tau_us), int(delta_us)
    return p


def dispatches_to_array(disp, n: int) -> np.ndarray:
    """Structured numpy array of the dispatch records held (at most n)."""
    dt = np.dtype([(f, np.int64) for f in DISPATCH_FIELDS])
    n = min(n, len(disp))
    out = np.zeros(n, dtype=dt)
    for i in range(n):
        for f in DISPATCH_FIELDS:
            out[f][i] = getattr(disp[i], f)
    return out


def greedy_decide(batch_sizes, cost_us, tau_us: int, delta_us: int, queue_len: int, oldest_wait_us: int) -> int:
    lib = load_library()
    keep = []
    p = make_policy(batch_sizes, cost_us, tau_us, delta_us, keep)
    b = C.c_int32(0)
    _check(lib.rafiki_greedy_decide(C.byref(p), queue_len, oldest_wait_us, C.byref(b)))
    return b.value


def greedy_simulate(arrival_us, batch_sizes, cost_us, tau_us: int, delta_us: int, cap: Optional[int] = None):
    """Host simulation of one model under the greedy policy: (latency_us, dispatches,
    total number of dispatches); at most ``cap`` dispatch records are returned."""
    lib = load_library()
    keep = []
    p = make_policy(batch_sizes, cost_us, tau_us, delta_us, keep)
    a = np.ascontiguousarray(arrival_us, dtype=np.int64)
    lat = np.zeros(a.size, dtype=np.int64)
    cap = a.size + 1 if cap is None else cap
    disp = (RafikiDispatch * max(cap, 1))()
    nd = C.c_int64(0)
    _check(lib.rafiki_greedy_simulate(C.byref(p), _i64p(a), a.size, _i64p(lat), disp if cap else None, cap,
                                      C.byref(nd)))
    return lat, dispatches_to_array(disp, min(nd.value, cap)), nd.value


def greedy_simulate_multi(arrival_us, policies):
    """Host simulation of independent servers sharing the queue; ``policies`` is a list
    of (batch_sizes, cost_us, tau_us, delta_us).  Returns (latency_us, dispatches)."""
    lib = load_library()
    keep = []
    pols = (RafikiGreedyPolicy * len(policies))()
    for k, p in enumerate(policies):
        pols[k] = make_policy(*p, keep)
    a = np.ascontiguousarray(arrival_us, dtype=np.int64)
    lat = np.zeros(a.size, dtype=np.int64)
    cap = a.size + 1
    disp = (RafikiDispatch * cap)()
    nd = C.c_int64(0)
    _check(lib.rafiki_greedy_simulate_multi(pols, len(policies), _i64p(a), a.size, _i64p(lat), disp, cap,
                                            C.byref(nd)))
    return lat, dispatches_to_array(disp, nd.value)


def _f64p(a: np.ndarray):
    return a.ctypes.data_as(C.POINTER(C.c_double))


class RLScheduler:
    """Handle over rafiki_rl_*: the actor-critic batch-size and model-subset scheduler."""

    def __init__(self, batch_sizes, cost_us, accuracy, tau_us: int, beta: float, queue_features: int = 128,
                 hidden: int = 64, seed: int = 0):
        lib = load_library()
        cost = np.ascontiguousarray(cost_us, dtype=np.int64)
        self._B = np.ascontiguousarray(batch_sizes, dtype=np.int32)
        self._cost = np.ascontiguousarray(cost.reshape(-1))
        self._acc = np.ascontiguousarray(accuracy, dtype=np.float64)
        cfg = RafikiRLConfig()
        cfg.n_models, cfg.n_sizes = cost.shape[0], self._B.size
        cfg.batch_sizes, cfg.cost_us, cfg.accuracy = _i32p(self._B), _i64p(self._cost), _f64p(self._acc)
        cfg.tau_us, cfg.beta, cfg.queue_features, cfg.hidden = int(tau_us), float(beta), queue_features, hidden
        h = C.c_void_p()
        _check(lib.rafiki_rl_create(C.byref(cfg), seed, C.byref(h)))
        self._h, self._lib = h, lib
        d, a, n = C.c_int(), C.c_int(), C.c_int64()
        _check(lib.rafiki_rl_info(h, C.byref(d), C.byref(a), C.byref(n)))
        self.state_dim, self.n_actions, self.n_params = d.value, a.value, n.value

    def params(self) -> np.ndarray:
        out = np.zeros(self.n_params)
        _check(self._lib.rafiki_rl_get_params(self._h, _f64p(out), self.n_params))
        return out

    def set_params(self, theta):
        t = np.ascontiguousarray(theta, dtype=np.float64)
        _check(self._lib.rafiki_rl_set_params(self._h, _f64p(t), t.size))

    def forward(self, state):
        s = np.ascontiguousarray(state, dtype=np.float64)
        pi = np.zeros(self.n_actions)
        v = C.c_double()
        _check(self._lib.rafiki_rl_forward(self._h, _f64p(s), _f64p(pi), C.byref(v)))
        return pi, v.value

    def gradient(self, states, actions, returns, c_v: float, c_e: float) -> np.ndarray:
        S = np.ascontiguousarray(states, dtype=np.float64)
        A = np.ascontiguousarray(actions, dtype=np.int32)
        R = np.ascontiguousarray(returns, dtype=np.float64)
        g = np.zeros(self.n_params)
        _check(self._lib.rafiki_rl_gradient(self._h, _f64p(S), _i32p(A), _f64p(R), R.size, c_v, c_e, _f64p(g)))
        return g

    def adam_step(self, grad, lr: float):
        g = np.ascontiguousarray(grad, dtype=np.float64)
        _check(self._lib.rafiki_rl_adam_step(self._h, _f64p(g), lr))

    def run_episode(self, arrival_us, mode: str = "argmax", actions=None, seed: int = 0):
        """mode 'given' (actions), 'sample' or 'argmax'.  Returns a dict of numpy arrays:
        actions, rewards, states, times (per decision) and latency (per request)."""
        a = np.ascontiguousarray(arrival_us, dtype=np.int64)
        acts_in = np.ascontiguousarray(actions if actions is not None else [], dtype=np.int32)
        cap = a.size
        out_a = np.zeros(cap, dtype=np.int32)
        out_r = np.zeros(cap)
        out_s = np.zeros((cap, self.state_dim))
        out_t = np.zeros(cap, dtype=np.int64)
        lat = np.zeros(a.size, dtype=np.int64)
        steps = C.c_int64()
        m = {"given": 0, "sample": 1, "argmax": 2}[mode]
        _check(self._lib.rafiki_rl_run_episode(self._h, _i64p(a), a.size, m, _i32p(acts_in), acts_in.size, seed,
                                               _i32p(out_a), _f64p(out_r), _f64p(out_s), _i64p(out_t), cap,
                                               C.byref(steps), _i64p(lat)))
        k = steps.value
        return {"actions": out_a[:k], "rewards": out_r[:k], "states": out_s[:k], "times": out_t[:k],
                "latency": lat}

    def train(self, arrival_us, episodes: int, gamma: float = 0.99, lr: float = 1e-3, c_v: float = 0.5,
              c_e: float = 0.01, seed: int = 0) -> np.ndarray:
        a = np.ascontiguousarray(arrival_us, dtype=np.int64)
        out = np.zeros(episodes)
        _check(self._lib.rafiki_rl_train(self._h, _i64p(a), a.size, episodes, gamma, lr, c_v, c_e, seed,
                                         _f64p(out)))
        return out

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._lib.rafiki_rl_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def make_layers(spec, params, keep: list):
    """rafiki_layer array for a layer list (plain attribute access on each layer)."""
    arr = (RafikiLayer * len(spec.layers))()
    for i, (L, P) in enumerate(zip(spec.layers, params.layers)):
        r = arr[i]
        r.op, r.input, r.input2 = L.op, L.input, L.input2
        r.c_in, r.c_out, r.kh, r.kw, r.stride, r.pad = L.c_in, L.c_out, L.kh, L.kw, L.stride, L.pad
        r.relu = 1 if L.relu else 0
        r.weight = _fptr(P.weight, keep)
        r.bias = _fptr(P.bias if L.bias else None, keep)
        if L.bn:
            r.bn_gamma, r.bn_beta = _fptr(P.bn_gamma, keep), _fptr(P.bn_beta, keep)
            r.bn_mean, r.bn_var = _fptr(P.bn_mean, keep), _fptr(P.bn_var, keep)
            r.bn_eps = float(P.bn_eps)
    keep.append(arr)
    return arr


def _expect(t, shape, dtype, name):
    """Raise ValueError unless torch tensor ``t`` is a contiguous device tensor of that shape and dtype."""
    if not t.is_cuda or t.dtype != dtype or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{name}: expected a contiguous device tensor {tuple(shape)} of {dtype}, got "
                         f"{tuple(t.shape)} {t.dtype} on {t.device}"
                         f"{'' if t.is_contiguous() else ' (not contiguous)'}")


def _combine_io(logits, out, labels):
    import torch
    if logits.dim() != 3:
        raise ValueError("logits: expected [S, n, C]")
    S, n, C = logits.shape
    _expect(logits, (S, n, C), torch.float32, "logits")
    _expect(out, (n, C), torch.float32, "output")
    _expect(labels, (n,), torch.int32, "labels")
    return S, n, C


def combine_mean(logits, out_probs, out_labels, stream=None):
    """Standalone combine: logits [S, n, C] fp32 -> mean softmax [n, C], first-index argmax [n]."""
    S, n, C = _combine_io(logits, out_probs, out_labels)
    _check(load_library().rafiki_combine_mean(_ptr(logits), S, n, C, _ptr(out_probs), _ptr(out_labels),
                                              _stream(stream)))


def combine_vote(logits, out_votes, out_labels, stream=None):
    """Standalone majority vote over logits [S, n, C] fp32."""
    S, n, C = _combine_io(logits, out_votes, out_labels)
    _check(load_library().rafiki_combine_vote(_ptr(logits), S, n, C, _ptr(out_votes), _ptr(out_labels),
                                              _stream(stream)))


def maxpool_nhwc_bf16(x, y, k: int, stride: int, pad: int, stream=None):
    """Standalone max-pool over a bf16 NHWC tensor x [n, h, w, c] into y [n, ho, wo, c]."""
    import torch
    n, h, w, c = x.shape
    _expect(x, (n, h, w, c), torch.bfloat16, "x")
    _expect(y, (n, (h + 2 * pad - k) // stride + 1, (w + 2 * pad - k) // stride + 1, c), torch.bfloat16, "y")
    _check(load_library().rafiki_maxpool_nhwc_bf16(_ptr(x), _ptr(y), n, h, w, c, k, stride, pad, _stream(stream)))


def probe_mfma_bf16(blocks: int, iters: int, out, stream=None):
    """Register-resident bf16 MFMA loop: blocks x 4 wavefronts x iters x 8 x 32768 FLOP."""
    _check(load_library().rafiki_probe_mfma_bf16(blocks, iters, _ptr(out), _stream(stream)))


def probe_hbm_read(x, blocks: int, out, stream=None):
    """One streaming pass of 16-byte loads over the bytes of device tensor x."""
    _check(load_library().rafiki_probe_hbm_read(_ptr(x), x.numel() * x.element_size(), blocks, _ptr(out),
                                                 _stream(stream)))


# (waves, wave tile, workgroup tile, TM x TN MFMA blocks per wave) of each main-loop variant
MAINLOOP_VARIANTS = {0: (8, "64x128", "256x256", 8), 1: (4, "128x128", "256x256", 16),
                     2: (4, "64x64", "128x128", 4), 3: (8, "64x32", "128x128", 2)}


def probe_mainloop(variant: int, sync: bool, blocks: int, ktiles: int, out, stream=None):
    """The GEMM main loop without memory loads: LDS fragment reads and MFMAs, with
    (sync) or without each K tile's LDS writes and barrier.  FLOP per launch:
    blocks x waves x ktiles x 4 x (TM x TN) x 32768."""
    _check(load_library().rafiki_probe_mainloop(variant, 1 if sync else 0, blocks, ktiles, _ptr(out),
                                                _stream(stream)))


def global_avgpool_nhwc_bf16(x, y, stream=None):
    """Standalone global average pool over a bf16 NHWC tensor x [n, h, w, c] into y [n, c]."""
    import torch
    n, h, w, c = x.shape
    _expect(x, (n, h, w, c), torch.bfloat16, "x")
    _expect(y, (n, c), torch.bfloat16, "y")
    _check(load_library().rafiki_global_avgpool_nhwc_bf16(_ptr(x), _ptr(y), n, h, w, c, _stream(stream)))


def tile_configs():
    """The bf16 GEMM kernel's tile configurations: list of dicts {bm, bn, waves, stages, bk}."""
    lib = load_library()
    out = []
    while True:
        v = [C.c_int() for _ in range(5)]
        if lib.rafiki_tile_config(len(out), *[C.byref(x) for x in v]) != RAFIKI_OK:
            return out
        out.append(dict(zip(("bm", "bn", "waves", "stages", "bk"), (x.value for x in v))))


class Ensemble:
    """Handle over ``rafiki_ensemble_create`` .. ``rafiki_ensemble_destroy``."""

    def __init__(self, specs: Sequence, params: Sequence, precision: str = "bf16", max_batch: int = 64):
        lib = load_library()
        keep: list = []
        descs = (RafikiModelDesc * len(specs))()
        for i, (s, p) in enumerate(zip(specs, params)):
            arr = make_layers(s, p, keep)
            descs[i].n_layers = len(s.layers)
            descs[i].layers = C.cast(arr, C.POINTER(RafikiLayer))
            descs[i].n_classes = s.n_classes
        s0 = specs[0]
        opts = RafikiOpts()
        if len(s0.input_shape) == 3:
            opts.input_kind = RAFIKI_INPUT_IMAGE_NCHW_F32
            opts.c, opts.h, opts.w = s0.input_shape
        else:
            opts.input_kind = RAFIKI_INPUT_TOKENS_I32
            opts.c, opts.h, opts.w = 1, s0.input_shape[0], 1
            opts.vocab = s0.vocab
        opts.precision = RAFIKI_BF16 if precision == "bf16" else RAFIKI_FP32
        opts.max_batch = max_batch
        h = C.c_void_p()
        _check(lib.rafiki_ensemble_create(descs, len(specs), C.byref(opts), C.byref(h)))
        self._h = h
        self._lib = lib
        self.n_models = len(specs)
        self.n_classes = s0.n_classes
        self.max_batch = max_batch

    def infer(self, batch, n: int, mask: int, out_probs, out_labels, stream=None):
        _check(self._lib.rafiki_ensemble_infer(self._h, _ptr(batch), n, mask, _ptr(out_probs), _ptr(out_labels),
                                               _stream(stream)))

    def infer_vote(self, batch, n: int, mask: int, out_votes, out_labels, stream=None):
        """Majority-vote combine (Section 5.2): out_votes = vote fractions, ties to the
        lowest-numbered selected model's class."""
        _check(self._lib.rafiki_ensemble_infer_vote(self._h, _ptr(batch), n, mask, _ptr(out_votes),
                                                    _ptr(out_labels), _stream(stream)))

    def infer_noalloc(self, batch, n: int, mask: int, out_probs, out_labels, stream=None):
        """infer with the call's scratch in the library's static device array (no allocation)."""
        _check(self._lib.rafiki_ensemble_infer_noalloc(self._h, _ptr(batch), n, mask, _ptr(out_probs),
                                                       _ptr(out_labels), _stream(stream)))

    def model_logits(self, model: int, batch, n: int, out_logits, stream=None):
        _check(self._lib.rafiki_ensemble_model_logits(self._h, model, _ptr(batch), n, _ptr(out_logits),
                                                      _stream(stream)))

    def profile(self, batch, batch_sizes, mask: int, reps: int = 10, stream=None):
        """c(b) in microseconds for each candidate size (mask = 1 << m gives c(m, b))."""
        import torch
        B = np.ascontiguousarray(batch_sizes, dtype=np.int32)
        bmax = int(B.max())
        probs = torch.empty((bmax, self.n_classes), dtype=torch.float32, device="cuda")
        labels = torch.empty((bmax,), dtype=torch.int32, device="cuda")
        out = np.zeros(B.size, dtype=np.int64)
        _check(self._lib.rafiki_ensemble_profile(self._h, _ptr(batch), _i32p(B), B.size, mask, reps, _ptr(probs),
                                                 _ptr(labels), _i64p(out), _stream(stream)))
        return out

    def serve_greedy(self, requests, arrival_us, batch_sizes, cost_us, tau_us: int, delta_us: int, mask: int,
                     out_probs, out_labels, combine: str = "mean", stream=None):
        """Real-time greedy serving of resident requests; returns (latency_us, dispatches)."""
        a = np.ascontiguousarray(arrival_us, dtype=np.int64)
        keep = []
        pol = make_policy(batch_sizes, cost_us, tau_us, delta_us, keep)
        lat = np.zeros(a.size, dtype=np.int64)
        cap = a.size + 1
        disp = (RafikiDispatch * cap)()
        nd = C.c_int64(0)
        _check(self._lib.rafiki_ensemble_serve_greedy(self._h, _ptr(requests), _i64p(a), a.size, C.byref(pol), mask,
                                                      1 if combine == "vote" else 0, _ptr(out_probs),
                                                      _ptr(out_labels), _i64p(lat), disp, cap, C.byref(nd),
                                                      _stream(stream)))
        return lat, dispatches_to_array(disp, nd.value)

    def serve_greedy_async(self, requests, arrival_us, policies, mask: int, out_probs, out_labels, stream=None):
        """Asynchronous serving, one model per batch; ``policies`` maps model index ->
        (batch_sizes, cost_us, tau_us, delta_us).  Returns (latency_us, dispatches)."""
        a = np.ascontiguousarray(arrival_us, dtype=np.int64)
        keep = []
        pols = (RafikiGreedyPolicy * self.n_models)()
        for m in range(self.n_models):
            if m in policies:
                pols[m] = make_policy(*policies[m], keep)
        lat = np.zeros(a.size, dtype=np.int64)
        cap = a.size + 1
        disp = (RafikiDispatch * cap)()
        nd = C.c_int64(0)
        _check(self._lib.rafiki_ensemble_serve_greedy_async(self._h, _ptr(requests), _i64p(a), a.size, pols, mask,
                                                            _ptr(out_probs), _ptr(out_labels), _i64p(lat), disp, cap,
                                                            C.byref(nd), _stream(stream)))
        return lat, dispatches_to_array(disp, nd.value)

    def serve_rl(self, agent, requests, arrival_us, out_probs, out_labels, mode: str = "argmax", seed: int = 0,
                 stream=None):
        """Real-time serving with the actor-critic agent choosing (subset, batch size) per
        decision.  Returns a dict: latency (per request), dispatches, actions and states
        (per decision)."""
        a = np.ascontiguousarray(arrival_us, dtype=np.int64)
        lat = np.zeros(a.size, dtype=np.int64)
        cap = a.size + 1
        disp = (RafikiDispatch * cap)()
        acts = np.zeros(cap, dtype=np.int32)
        states = np.zeros((cap, agent.state_dim))
        steps = C.c_int64(0)
        _check(self._lib.rafiki_ensemble_serve_rl(self._h, agent._h, _ptr(requests), _i64p(a), a.size,
                                                  {"sample": 1, "argmax": 2}[mode], seed, _ptr(out_probs),
                                                  _ptr(out_labels), _i64p(lat), disp, _i32p(acts), _f64p(states),
                                                  cap, C.byref(steps), _stream(stream)))
        k = steps.value
        return {"latency": lat, "dispatches": dispatches_to_array(disp, k), "actions": acts[:k],
                "states": states[:k]}

    def trace(self, enable, concurrent: bool = False):
        """Per-launch timing on (models one after another, or concurrent=True: on their
        own streams in their kept schedule) or off."""
        _check(self._lib.rafiki_ensemble_trace(self._h, (2 if concurrent else 1) if enable else 0))

    def force_tile(self, cfg: int):
        """Use tile configuration ``cfg`` for every unsplit bf16 GEMM it suits (-1: tuned)."""
        _check(self._lib.rafiki_ensemble_force_tile(self._h, cfg))

    def get_schedule(self, n: int, mask: int):
        """Schedule kept for (n, mask): (solo, ascending).  solo -1: all models concurrent;
        m: model m alone on one lane, the others chained on a second lane, longest first
        (ascending 0) or shortest first (ascending 1)."""
        v, a = C.c_int(0), C.c_int(0)
        _check(self._lib.rafiki_ensemble_get_schedule(self._h, n, mask, C.byref(v), C.byref(a)))
        return v.value, a.value

    def set_schedule(self, n: int, mask: int, solo: int, ascending: int = 0):
        _check(self._lib.rafiki_ensemble_set_schedule(self._h, n, mask, solo, ascending))

    def get_schedule_pair(self, n: int, mask: int):
        """The pair (a, b) whose aligned layers the schedule kept for (n, mask) runs as
        two-member launches, or (-1, -1)."""
        a, b = C.c_int(0), C.c_int(0)
        _check(self._lib.rafiki_ensemble_get_schedule_pair(self._h, n, mask, C.byref(a), C.byref(b)))
        return a.value, b.value

    def set_schedule_pair(self, n: int, mask: int, a: int, b: int = -1):
        _check(self._lib.rafiki_ensemble_set_schedule_pair(self._h, n, mask, a, b))

    def get_schedule_tiles(self, n: int, mask: int) -> int:
        """Tile policy of the schedule kept for (n, mask): 0 the fastest tiles alone; 1 the
        layers with output maps of at most 14 x 14 pixels on their lean tiles; 2 as 1, and
        the model alone on its lane without the direct conv kernel (GEMM tiles)."""
        v = C.c_int(0)
        _check(self._lib.rafiki_ensemble_get_schedule_tiles(self._h, n, mask, C.byref(v)))
        return v.value

    def set_schedule_tiles(self, n: int, mask: int, lean: int):
        _check(self._lib.rafiki_ensemble_set_schedule_tiles(self._h, n, mask, lean))

    def pairing(self, a: int, b: int) -> int:
        """Number of aligned ops of models a < b (0: not pairable)."""
        v = C.c_int(0)
        _check(self._lib.rafiki_ensemble_pairing(self._h, a, b, C.byref(v)))
        return v.value

    def use_graphs(self, enable: bool):
        """Turn graph replay of the forward passes on or off (drops every kept graph)."""
        _check(self._lib.rafiki_ensemble_use_graphs(self._h, 1 if enable else 0))

    def graph_stats(self):
        """(graphs kept, replays so far, failed captures)."""
        g, r, f = C.c_int(0), C.c_longlong(0), C.c_longlong(0)
        _check(self._lib.rafiki_ensemble_graph_stats(self._h, C.byref(g), C.byref(r), C.byref(f)))
        return g.value, r.value, f.value

    def trace_read(self):
        """List of dicts {kind, model, layer, flops, bytes, ms, tile_cfg, splits} for the traced launches."""
        cnt = C.c_int(0)
        _check(self._lib.rafiki_ensemble_trace_read(self._h, None, 0, C.byref(cnt)))
        buf = (RafikiTraceRec * max(cnt.value, 1))()
        _check(self._lib.rafiki_ensemble_trace_read(self._h, buf, cnt.value, C.byref(cnt)))
        return [{"kind": KERNEL_CLASSES[r.kind], "model": r.model, "layer": r.layer, "flops": r.flops,
                 "bytes": r.bytes, "ms": r.ms, "tile_cfg": r.tile_cfg, "splits": r.splits}
                for r in buf[:cnt.value]]

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            _check(self._lib.rafiki_ensemble_destroy(self._h))
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

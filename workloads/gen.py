"""Seeded draws for the synthetic workloads.

Every array is drawn from ``numpy.random.Generator(PCG64(seed))``.  Model k of a
configuration uses seed k (1-based, in configuration order); request batches use
seed 0.  Parameters are drawn layer by layer in layer order, within a layer as
weight, then batch-norm running mean, then running variance (biases are zero and
BN gamma/beta are 1/0, so they consume no draws).

Distributions:
* conv / FC / conv1d weights: He normal, standard deviation sqrt(2 / fan_in)
  (float32 standard-normal draws scaled by that deviation);
* embedding tables: normal, standard deviation 0.1 (same construction);
* BN running statistics: mean ~ N(0, 0.1) (0.1 is the standard deviation),
  variance ~ U(0.5, 1.5); or the identity (mean 0, variance 1);
* images: U[0, 1] or N(0, 1); token ids: uniform integers in [0, vocab).

For bf16 workloads each drawn weight, table and image is rounded once,
round-to-nearest-even, to a bfloat16-representable float32: those values *are*
the model and the request.  Nothing here computes any step of the inference.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional, Tuple

import numpy as np

from .specs import (ModelSpec, Layer, CONV2D, FC, EMBEDDING, CONV1D_MAXTIME, toy_cnn,
                    resnet20, resnet50, resnet101, vgg16, textcnn)

BN_EPS = 1e-5


def round_bf16_rne_f32(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32.

    Works on the IEEE bit pattern: add 0x7FFF plus the lowest kept bit, then clear
    the low 16 bits.  Inputs here are finite.
    """
    u = np.array(a, dtype=np.float32, copy=True).view(np.uint32)
    lsb = u >> 16
    lsb &= 1
    u += np.uint32(0x7FFF)      # finite inputs: no uint32 overflow (max 0xFF7FFFFF + 0x8000)
    u += lsb
    u &= np.uint32(0xFFFF0000)
    return u.view(np.float32)


@dataclass
class LayerParams:
    weight: Optional[np.ndarray] = None     # float32, canonical layout
    bias: Optional[np.ndarray] = None       # float32 [c_out]
    bn_gamma: Optional[np.ndarray] = None
    bn_beta: Optional[np.ndarray] = None
    bn_mean: Optional[np.ndarray] = None
    bn_var: Optional[np.ndarray] = None
    bn_eps: float = BN_EPS


@dataclass
class ModelParams:
    spec: ModelSpec
    layers: List[LayerParams]
    seed: int
    bf16: bool


def gen_params(spec: ModelSpec, seed: int, bf16: bool, bn_kind: str = "random") -> ModelParams:
    """Draw the parameters of ``spec`` from ``PCG64(seed)``.  ``bn_kind`` is
    ``"random"`` (mean ~ N(0, 0.1), var ~ U(0.5, 1.5)) or ``"identity"``."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out: List[LayerParams] = []
    for L in spec.layers:
        p = LayerParams()
        if L.op == EMBEDDING:
            w = rng.standard_normal(size=L.weight_shape(), dtype=np.float32)
            w *= np.float32(0.1)
            p.weight = round_bf16_rne_f32(w) if bf16 else w
        elif L.has_weight():
            w = rng.standard_normal(size=L.weight_shape(), dtype=np.float32)
            w *= np.float32(np.sqrt(2.0 / L.fan_in()))
            p.weight = round_bf16_rne_f32(w) if bf16 else w
        if L.bias:
            p.bias = np.zeros(L.c_out, dtype=np.float32)
        if L.bn:
            p.bn_gamma = np.ones(L.c_out, dtype=np.float32)
            p.bn_beta = np.zeros(L.c_out, dtype=np.float32)
            if bn_kind == "random":
                p.bn_mean = rng.normal(0.0, 0.1, size=L.c_out).astype(np.float32)
                p.bn_var = rng.uniform(0.5, 1.5, size=L.c_out).astype(np.float32)
            elif bn_kind == "identity":
                p.bn_mean = np.zeros(L.c_out, dtype=np.float32)
                p.bn_var = np.ones(L.c_out, dtype=np.float32)
            else:
                raise ValueError(bn_kind)
        out.append(p)
    return ModelParams(spec, out, seed, bf16)


def gen_images(n: int, shape: Tuple[int, int, int], dist: str, bf16: bool, seed: int = 0) -> np.ndarray:
    """Request batch of images, NCHW float32.  ``dist`` is ``"uniform"`` (U[0,1]) or ``"normal"``."""
    rng = np.random.Generator(np.random.PCG64(seed))
    if dist == "uniform":
        x = rng.random(size=(n,) + tuple(shape), dtype=np.float32)
    elif dist == "normal":
        x = rng.standard_normal(size=(n,) + tuple(shape), dtype=np.float32)
    else:
        raise ValueError(dist)
    return round_bf16_rne_f32(x) if bf16 else x


def gen_tokens(n: int, seq_len: int, vocab: int, seed: int = 0) -> np.ndarray:
    """Request batch of token-id sequences, int32 ``[n, seq_len]``, uniform in [0, vocab)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.integers(0, vocab, size=(n, seq_len), dtype=np.int32)


@dataclass
class Config:
    cid: int
    name: str
    models: List[Callable[[], ModelSpec]]
    seeds: List[int]
    n: int
    precision: str            # "fp32" or "bf16"
    bn_kind: str              # "identity" or "random"
    input_dist: str           # "uniform", "normal" or "tokens"
    batches: List[int] = field(default_factory=list)     # batch sizes of a sweep
    masks: List[int] = field(default_factory=list)       # subset masks of a sweep

    @property
    def bf16(self) -> bool:
        return self.precision == "bf16"


CONFIGS: Dict[int, Config] = {
    1: Config(1, "toy_fp32", [toy_cnn, toy_cnn], [1, 2], 8, "fp32", "identity", "uniform"),
    2: Config(2, "resnet20x3", [resnet20, resnet20, resnet20], [1, 2, 3], 128, "bf16", "random", "uniform"),
    3: Config(3, "r50_vgg16_r101", [resnet50, vgg16, resnet101], [1, 2, 3], 64, "bf16", "random", "normal"),
    4: Config(4, "r50_vgg16_r101_sweep", [resnet50, vgg16, resnet101], [1, 2, 3], 256, "bf16", "random",
              "normal", batches=[1, 4, 16, 64, 256], masks=[0b001, 0b011, 0b111]),
    5: Config(5, "textcnn_x4", [textcnn, textcnn, textcnn, textcnn], [1, 2, 3, 4], 512, "bf16", "random",
              "tokens"),
}


def build_config(cid: int, n: Optional[int] = None, models: Optional[List[int]] = None):
    """Specs, parameters and request batch of configuration ``cid``.

    ``models`` optionally restricts which members are drawn (indices into the
    configuration's model list; each keeps its own seed).  Returns
    ``(config, specs, params, batch)``."""
    cfg = CONFIGS[cid]
    n = cfg.n if n is None else n
    idx = list(range(len(cfg.models))) if models is None else list(models)
    specs = [cfg.models[i]() for i in idx]
    params = [gen_params(s, cfg.seeds[i], cfg.bf16, cfg.bn_kind) for s, i in zip(specs, idx)]
    s0 = specs[0]
    if cfg.input_dist == "tokens":
        batch = gen_tokens(n, s0.input_shape[0], s0.vocab)
    else:
        batch = gen_images(n, s0.input_shape, cfg.input_dist, cfg.bf16)
    return cfg, specs, params, batch

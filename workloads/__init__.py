"""Seeded synthetic workloads: model architectures as plain layer lists, and the
random draws (parameters, request batches) that both the oracle and the HIP path
consume as data, and the seeded request-arrival process of the serving experiments.

Nothing in this package computes any part of the inference method: it only
describes networks and draws numbers from seeded generators.
"""
from .specs import (Layer, toy_cnn, resnet20, resnet_cifar, resnet50, resnet101, vgg16, textcnn,
                    ModelSpec, CONV2D, MAXPOOL2D, GLOBAL_AVGPOOL, FC, EMBEDDING,
                    CONV1D_MAXTIME, CONCAT, OP_NAMES)
from .gen import (ModelParams, gen_params, gen_images, gen_tokens, round_bf16_rne_f32,
                  CONFIGS, Config, build_config)
from .arrivals import sine_coefficients, sine_rate, sine_arrivals

__all__ = [
    "Layer", "ModelSpec", "toy_cnn", "resnet20", "resnet_cifar", "resnet50", "resnet101", "vgg16", "textcnn",
    "CONV2D", "MAXPOOL2D", "GLOBAL_AVGPOOL", "FC", "EMBEDDING", "CONV1D_MAXTIME", "CONCAT",
    "OP_NAMES", "ModelParams", "gen_params", "gen_images", "gen_tokens", "round_bf16_rne_f32",
    "CONFIGS", "Config", "build_config", "sine_coefficients", "sine_rate", "sine_arrivals",
]

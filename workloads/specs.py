"""Network architectures of the ensemble members, as topologically ordered layer lists.

The paper names the model families its inference service deploys (ResNets, VGGs,
Inception, ...; Section 3, the ConvNet comparison, and the built-in task table) and
text models for sentiment analysis, but it defines no architecture.  The layer lists
below are the textbook definitions of the families the benchmark configurations name:

* a two-conv toy CNN (CIFAR-shaped),
* ResNet-20 (He et al. 2016, CIFAR variant; projection shortcuts),
* ResNet-50 / ResNet-101 v1.5 (bottleneck blocks, stride on the 3x3 conv),
* VGG-16 configuration D,
* a Kim-style TextCNN (embedding, conv1d widths 3/4/5 with 100 filters, max over time).

Tensor ids: layer i writes tensor i; id -1 is the model input.  ``input2`` of a
CONV2D names a residual tensor added before the ReLU.  ``input``/``input2`` of a
CONCAT name the two tensors joined along the channel axis (first, then second).
Parameter layouts are canonical: conv OIHW ``[c_out, c_in, kh, kw]``, FC
``[c_out, c_in]`` (when its input is spatial, ``c_in`` is indexed in (c, h, w)
order), conv1d ``[c_out, c_in, kw]``, embedding ``[vocab, dim]``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

# Operation codes; the numeric values match the C header's enum.
CONV2D = 1
MAXPOOL2D = 2
GLOBAL_AVGPOOL = 3
FC = 4
EMBEDDING = 5
CONV1D_MAXTIME = 6
CONCAT = 7
OP_NAMES = {CONV2D: "conv2d", MAXPOOL2D: "maxpool2d", GLOBAL_AVGPOOL: "global_avgpool",
            FC: "fc", EMBEDDING: "embedding", CONV1D_MAXTIME: "conv1d_maxtime", CONCAT: "concat"}


@dataclass
class Layer:
    op: int
    input: int = -1
    input2: int = -1
    c_in: int = 0
    c_out: int = 0
    kh: int = 1
    kw: int = 1
    stride: int = 1
    pad: int = 0
    relu: bool = False
    bias: bool = False     # layer has a bias vector
    bn: bool = False       # layer is followed by inference batch-norm (gamma, beta, mean, var)

    def has_weight(self) -> bool:
        return self.op in (CONV2D, FC, EMBEDDING, CONV1D_MAXTIME)

    def weight_shape(self) -> Tuple[int, ...]:
        if self.op == CONV2D:
            return (self.c_out, self.c_in, self.kh, self.kw)
        if self.op == FC:
            return (self.c_out, self.c_in)
        if self.op == CONV1D_MAXTIME:
            return (self.c_out, self.c_in, self.kw)
        if self.op == EMBEDDING:
            return (self.c_in, self.c_out)
        raise ValueError("layer has no weight")

    def fan_in(self) -> int:
        if self.op == CONV2D:
            return self.c_in * self.kh * self.kw
        if self.op == FC:
            return self.c_in
        if self.op == CONV1D_MAXTIME:
            return self.c_in * self.kw
        raise ValueError("layer has no fan-in")


@dataclass
class ModelSpec:
    name: str
    layers: List[Layer]
    n_classes: int
    input_shape: Tuple[int, ...]          # (C, H, W) for images, (L,) for token sequences
    vocab: int = 0

    def param_count(self, count_bn_affine: bool = True) -> int:
        """Number of trainable scalars: weights, biases and (optionally) BN gamma/beta."""
        total = 0
        for L in self.layers:
            if L.has_weight():
                n = 1
                for d in L.weight_shape():
                    n *= d
                total += n
            if L.bias:
                total += L.c_out
            if L.bn and count_bn_affine:
                total += 2 * L.c_out
        return total


class _Builder:
    def __init__(self):
        self.layers: List[Layer] = []

    def add(self, **kw) -> int:
        self.layers.append(Layer(**kw))
        return len(self.layers) - 1

    def conv(self, x, c_in, c_out, k, stride=1, pad=None, relu=True, bn=True, bias=False, residual=-1):
        if pad is None:
            pad = k // 2
        return self.add(op=CONV2D, input=x, input2=residual, c_in=c_in, c_out=c_out, kh=k, kw=k,
                        stride=stride, pad=pad, relu=relu, bn=bn, bias=bias)


def toy_cnn() -> ModelSpec:
    """conv3x3(3->16)+BN+ReLU, maxpool 2x2/2, conv3x3(16->32)+BN+ReLU, GAP, FC(32->10)."""
    b = _Builder()
    x = b.conv(-1, 3, 16, 3)
    x = b.add(op=MAXPOOL2D, input=x, c_in=16, c_out=16, kh=2, kw=2, stride=2, pad=0)
    x = b.conv(x, 16, 32, 3)
    x = b.add(op=GLOBAL_AVGPOOL, input=x, c_in=32, c_out=32)
    b.add(op=FC, input=x, c_in=32, c_out=10, bias=True)
    return ModelSpec("toy_cnn", b.layers, 10, (3, 32, 32))


def resnet20() -> ModelSpec:
    """CIFAR ResNet-20: 3 stages x 3 basic blocks at widths 16/32/64.

    The first block of stages 2 and 3 strides by 2 and uses a 1x1 stride-2 conv + BN
    projection shortcut.  Within a block the layer order is [projection], conv_a, conv_b.
    """
    return resnet_cifar(3)


def resnet_cifar(blocks: int, widths: Tuple[int, int, int] = (16, 32, 64), n_classes: int = 10,
                 name: Optional[str] = None) -> ModelSpec:
    """CIFAR ResNet of 6 * blocks + 2 layers (blocks = 3: ResNet-20, 5: ResNet-32, ...),
    the stem and first stage at widths[0], stages 2 and 3 at widths[1] and widths[2]."""
    b = _Builder()
    x = b.conv(-1, 3, widths[0], 3)
    c_prev = widths[0]
    for stage, width in enumerate(widths):
        for blk in range(blocks):
            stride = 2 if (stage > 0 and blk == 0) else 1
            if stride != 1 or c_prev != width:
                sc = b.conv(x, c_prev, width, 1, stride=stride, pad=0, relu=False)
            else:
                sc = x
            a = b.conv(x, c_prev, width, 3, stride=stride)
            x = b.conv(a, width, width, 3, relu=True, residual=sc)
            c_prev = width
    x = b.add(op=GLOBAL_AVGPOOL, input=x, c_in=c_prev, c_out=c_prev)
    b.add(op=FC, input=x, c_in=c_prev, c_out=n_classes, bias=True)
    return ModelSpec(name or f"resnet{6 * blocks + 2}", b.layers, n_classes, (3, 32, 32))


def _resnet_bottleneck(name: str, blocks: Tuple[int, int, int, int]) -> ModelSpec:
    """ResNet v1.5 with bottleneck blocks (the stride sits on the 3x3 conv).

    Within a block the layer order is [projection], 1x1 reduce, 3x3, 1x1 expand; the
    projection (1x1 stride-s conv + BN) exists on the first block of each stage.
    """
    b = _Builder()
    x = b.conv(-1, 3, 64, 7, stride=2, pad=3)
    x = b.add(op=MAXPOOL2D, input=x, c_in=64, c_out=64, kh=3, kw=3, stride=2, pad=1)
    c_prev = 64
    for stage, (nb, width) in enumerate(zip(blocks, (64, 128, 256, 512))):
        for blk in range(nb):
            stride = 2 if (stage > 0 and blk == 0) else 1
            if blk == 0:
                sc = b.conv(x, c_prev, 4 * width, 1, stride=stride, pad=0, relu=False)
            else:
                sc = x
            a = b.conv(x, c_prev, width, 1, pad=0)
            a = b.conv(a, width, width, 3, stride=stride, pad=1)
            x = b.conv(a, width, 4 * width, 1, pad=0, relu=True, residual=sc)
            c_prev = 4 * width
    x = b.add(op=GLOBAL_AVGPOOL, input=x, c_in=2048, c_out=2048)
    b.add(op=FC, input=x, c_in=2048, c_out=1000, bias=True)
    return ModelSpec(name, b.layers, 1000, (3, 224, 224))


def resnet50() -> ModelSpec:
    return _resnet_bottleneck("resnet50", (3, 4, 6, 3))


def resnet101() -> ModelSpec:
    return _resnet_bottleneck("resnet101", (3, 4, 23, 3))


def vgg16() -> ModelSpec:
    """VGG-16 configuration D: 13 conv3x3 (pad 1, bias, ReLU), 5 max-pools 2x2/2,
    FC 25088->4096->4096->1000 (bias; ReLU on the first two; dropout is identity)."""
    b = _Builder()
    x, c_prev = -1, 3
    for item in (64, 64, "M", 128, 128, "M", 256, 256, 256, "M", 512, 512, 512, "M", 512, 512, 512, "M"):
        if item == "M":
            x = b.add(op=MAXPOOL2D, input=x, c_in=c_prev, c_out=c_prev, kh=2, kw=2, stride=2, pad=0)
        else:
            x = b.conv(x, c_prev, item, 3, bn=False, bias=True)
            c_prev = item
    x = b.add(op=FC, input=x, c_in=512 * 7 * 7, c_out=4096, bias=True, relu=True)
    x = b.add(op=FC, input=x, c_in=4096, c_out=4096, bias=True, relu=True)
    b.add(op=FC, input=x, c_in=4096, c_out=1000, bias=True)
    return ModelSpec("vgg16", b.layers, 1000, (3, 224, 224))


def textcnn(vocab: int = 30000, seq_len: int = 256, dim: int = 300, filters: int = 100,
            widths=(3, 4, 5), n_classes: int = 2) -> ModelSpec:
    """Embedding -> for each width w: valid conv1d(dim->filters, w) + bias + ReLU + max over
    time -> concatenate in width order -> FC(filters*len(widths) -> n_classes)."""
    b = _Builder()
    e = b.add(op=EMBEDDING, input=-1, c_in=vocab, c_out=dim)
    feats = [b.add(op=CONV1D_MAXTIME, input=e, c_in=dim, c_out=filters, kh=1, kw=w,
                   relu=True, bias=True) for w in widths]
    x, c = feats[0], filters
    for f in feats[1:]:
        x = b.add(op=CONCAT, input=x, input2=f, c_in=c, c_out=c + filters)
        c += filters
    b.add(op=FC, input=x, c_in=c, c_out=n_classes, bias=True)
    return ModelSpec("textcnn", b.layers, n_classes, (seq_len,), vocab=vocab)

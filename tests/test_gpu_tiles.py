"""Every tile configuration of the bf16 GEMM kernel gives bitwise-identical results.

The tuner picks, per layer and batch size, the fastest configuration; that is only
sound if the choice never changes a bit.  Each probe model is a convolution (unsplit,
or split over K where the shape asks for it: the split itself is fixed by the shape,
and the forced configuration is the one launched), followed by
global average pooling and a random FC: a change of any single conv output element
moves the pooled sum by far more than its fp32 rounding, so equal logits mean equal
conv outputs.  The logits are also checked against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from workloads import Layer, ModelSpec, CONV2D, GLOBAL_AVGPOOL, FC
from paper_1804_06087_amd import Ensemble
from paper_1804_06087_amd.binding import tile_configs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def conv(i, c_in, c_out, k, s=1, relu=True, res=-1):
    return Layer(op=CONV2D, input=i, input2=res, c_in=c_in, c_out=c_out, kh=k, kw=k, stride=s, pad=k // 2,
                 relu=relu, bn=True)


def fits(bn, c_out):
    """The runtime's rule for which channel tiles suit a layer."""
    if c_out <= 32:
        return bn == 32
    if c_out <= 64:
        return bn <= 64
    return 64 <= bn <= -(-c_out // 64) * 64


CASES = {
    # name: (conv layers, input (C, H, W), n)
    # 64 storage channels: K ordered (channel block, tap, channel); ragged M
    "aligned_3x3_cout256": ([conv(-1, 64, 256, 3)], (64, 20, 20), 21),
    # 24 channels: K ordered (tap, channel) with per-lane decode; ragged N tile
    "unaligned_3x3_cout96": ([conv(-1, 24, 96, 3)], (24, 20, 20), 41),
    # 32-channel tiles
    "unaligned_3x3_cout32": ([conv(-1, 16, 32, 3)], (16, 24, 24), 29),
    # residual add after a stride-2 3x3, projection shortcut
    "residual_s2_cout128": ([conv(-1, 64, 128, 1, s=2, relu=False), conv(-1, 64, 128, 3, s=2, res=0)],
                            (64, 32, 32), 65),
    # residual add after a stride-1 3x3, rows of 18 pixels
    "residual_s1_cout128": ([conv(-1, 64, 128, 1, relu=False), conv(-1, 64, 128, 3, res=0)], (64, 12, 18), 76),
    # 7x7 images: every tile spans several images
    "aligned_3x3_7x7": ([conv(-1, 128, 128, 3)], (128, 7, 7), 340),
    # few output rows and a long K: split over K (the split is fixed by the shape, the
    # tile is not), residual added in the split-K reduction
    "split_k_3x3_7x7_residual": ([conv(-1, 512, 256, 1, relu=False), conv(-1, 512, 256, 3, res=0)], (512, 7, 7), 4),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_all_tile_configs_bitwise_equal(name):
    layers, shape, n = CASES[name]
    L = list(layers)
    c_out = L[-1].c_out
    L.append(Layer(op=GLOBAL_AVGPOOL, input=len(L) - 1, c_in=c_out, c_out=c_out))
    L.append(Layer(op=FC, input=len(L) - 1, c_in=c_out, c_out=10, bias=True))
    spec = ModelSpec("tiles", L, 10, shape)
    params = wl.gen_params(spec, 7, True, "random")
    batch = wl.gen_images(n, shape, "normal", True, seed=13)
    cfgs = tile_configs()
    assert len(cfgs) >= 2
    x = torch.from_numpy(batch).to(DEV)
    out = torch.empty((n, 10), dtype=torch.float32, device=DEV)
    results = {}
    with Ensemble([spec], [params], precision="bf16", max_batch=n) as ens:
        for i, c in enumerate(cfgs):
            if not all(fits(c["bn"], lay.c_out) for lay in layers):
                continue
            ens.force_tile(i)
            out.fill_(float("nan"))
            ens.model_logits(0, x, n, out)
            torch.cuda.synchronize()
            results[i] = out.cpu().numpy().copy()
        ens.force_tile(-1)
    assert len(results) >= 2, "fewer than two configurations suit the probe"
    ref_cfg = min(results)
    for i, z in results.items():
        assert np.isfinite(z).all(), (i, cfgs[i])
        assert np.array_equal(z.view(np.uint32), results[ref_cfg].view(np.uint32)), (i, cfgs[i])
    ref = oracle.run_model(spec, params, batch, act="bf16")
    z = results[ref_cfg]
    err = np.abs(z - ref).max() / np.abs(ref).max()
    assert err <= 1e-2, err

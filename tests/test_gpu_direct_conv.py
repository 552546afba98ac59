"""The direct conv kernel (weights and an input patch per 16 x 16 output tile held in
LDS) gives the same bits as the bf16 GEMM kernel.

The tuner times it as one more candidate of the layers it takes (no residual; 3x3
stride 1 from 64 to 64 or 128 channels, optionally with the fused 2x2 max-pool, or with
64 output channels and ReLU 3x3 stride 1 and 7x7 stride 2 over the 8 storage channels
of an image), so its results must not depend on the choice.  Each probe model ends in
global average pooling and a random FC, as in the tile tests: equal logits mean equal
conv outputs.  Covered: maps that are not multiples of the 16 x 16 tile (ragged tiles in
both directions, odd sizes), fewer tiles than compute units and many tiles per
workgroup, the fused pool after a 3 -> 64 first layer, 7x7 stride-2 stems on odd sizes,
64 -> 128 channels as two halves (also pooled), the pool on ragged tiles with and
without ReLU, a 64 -> 64 layer after a strided one,
and layers the kernel does not take (residual; an RGB layer without ReLU) next to ones
it does.  Also against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from workloads import Layer, ModelSpec, CONV2D, MAXPOOL2D, GLOBAL_AVGPOOL, FC
from paper_1804_06087_amd import Ensemble, RAFIKI_TILE_DIRECT
from paper_1804_06087_amd.binding import tile_configs

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def conv(i, c_in, c_out, k, s=1, relu=True, res=-1):
    return Layer(op=CONV2D, input=i, input2=res, c_in=c_in, c_out=c_out, kh=k, kw=k, stride=s, pad=k // 2,
                 relu=relu, bn=True)


def pool(i, c):
    return Layer(op=MAXPOOL2D, input=i, c_in=c, c_out=c, kh=2, kw=2, stride=2, pad=0)


CASES = {
    # name: (layers, input (C, H, W), n, number of layers the direct kernel takes)
    "ragged_20x36": ([conv(-1, 64, 64, 3)], (64, 20, 36), 5, 1),
    "odd_15x17": ([conv(-1, 64, 64, 3)], (64, 15, 17), 3, 1),
    "many_tiles_per_workgroup": ([conv(-1, 64, 64, 3)], (64, 32, 32), 300, 1),
    "fused_pool_after_rgb": ([conv(-1, 3, 64, 3), conv(0, 64, 64, 3), pool(1, 64)], (3, 36, 28), 17, 2),
    # the 8 storage channels of an RGB image: 3x3 stride 1, 7x7 stride 2 (stems, odd sizes)
    "rgb_3x3_many_tiles": ([conv(-1, 3, 64, 3)], (3, 40, 48), 90, 1),
    "stem_7x7_s2_odd": ([conv(-1, 3, 64, 7, s=2)], (3, 45, 38), 5, 1),
    "stem_7x7_s2_many_tiles": ([conv(-1, 3, 64, 7, s=2)], (3, 64, 64), 300, 1),
    # without ReLU the 8-channel layers stay on the GEMM; the 64-channel one does not care
    "rgb_no_relu_then_64": ([conv(-1, 3, 64, 3, relu=False), conv(0, 64, 64, 3, relu=False)], (3, 20, 20), 4, 1),
    # 64 -> 128 channels: two workgroups per tile, one per 64-channel half (also pooled)
    "cout128_ragged": ([conv(-1, 64, 128, 3)], (64, 20, 36), 7, 1),
    "cout128_pool_many_tiles": ([conv(-1, 64, 128, 3), pool(0, 128)], (64, 32, 32), 200, 1),
    "after_stride2_and_residual_next": ([conv(-1, 64, 64, 3, s=2), conv(0, 64, 64, 3), conv(1, 64, 64, 3, res=0)],
                                        (64, 34, 40), 6, 1),
    "relu_off_two_layers": ([conv(-1, 64, 64, 3, relu=False), conv(0, 64, 64, 3)], (64, 18, 16), 9, 2),
    # the fused pool on ragged tiles, with ReLU (maximum on the bit patterns) and without
    "pool_ragged_many_tiles": ([conv(-1, 64, 64, 3), pool(0, 64)], (64, 36, 52), 40, 1),
    "pool_no_relu_ragged": ([conv(-1, 64, 64, 3, relu=False), pool(0, 64)], (64, 20, 36), 6, 1),
    # an image smaller than one tile, pooled
    "tiny_4x6_pool": ([conv(-1, 64, 64, 3), pool(0, 64)], (64, 4, 6), 3, 1),
}


def build(layers, shape):
    L = list(layers)
    c = L[-1].c_out
    L.append(Layer(op=GLOBAL_AVGPOOL, input=len(L) - 1, c_in=c, c_out=c))
    L.append(Layer(op=FC, input=len(L) - 1, c_in=c, c_out=10, bias=True))
    return ModelSpec("direct_conv", L, 10, shape)


def logits_and_tiles(ens, x, n):
    out = torch.full((n, 10), float("nan"), dtype=torch.float32, device=DEV)
    ens.trace(True)
    ens.model_logits(0, x, n, out)
    torch.cuda.synchronize()
    recs = ens.trace_read()
    ens.trace(False)
    return out.cpu().numpy().copy(), [r["tile_cfg"] for r in recs if r["kind"] == "conv_mfma"]


@pytest.mark.parametrize("name", sorted(CASES))
def test_direct_conv_bitwise_equal_to_gemm(name):
    layers, shape, n, n_direct = CASES[name]
    spec = build(layers, shape)
    params = wl.gen_params(spec, 5, True, "random")
    batch = wl.gen_images(n, shape, "normal", True, seed=3)
    x = torch.from_numpy(batch).to(DEV)
    direct_id = len(tile_configs())   # the trace's tile id of the direct kernel
    with Ensemble([spec], [params], precision="bf16", max_batch=n) as ens:
        ens.force_tile(RAFIKI_TILE_DIRECT)
        zd, tiles = logits_and_tiles(ens, x, n)
        assert tiles.count(direct_id) == n_direct, tiles
        results = {"direct": zd}
        for i, c in enumerate(tile_configs()):   # GEMM tiles with 64-wide channel tiles
            if c["bn"] != 64:
                continue
            ens.force_tile(i)
            z, tiles = logits_and_tiles(ens, x, n)
            assert direct_id not in tiles
            results[i] = z
        ens.force_tile(-1)
        results["tuned"], _ = logits_and_tiles(ens, x, n)
    assert len(results) >= 3
    for k, z in results.items():
        assert np.isfinite(z).all(), k
        assert np.array_equal(z.view(np.uint32), zd.view(np.uint32)), k
    ref = oracle.run_model(spec, params, batch, act="bf16")
    err = np.abs(zd - ref).max() / np.abs(ref).max()
    assert err <= 1e-2, err


def test_force_direct_rejects_nothing_and_restores():
    """Forcing the direct kernel on a model with no layer it takes changes nothing;
    -1 restores the tuned choice; unknown ids are refused."""
    from paper_1804_06087_amd import RafikiError
    spec = build([conv(-1, 32, 96, 3)], (32, 12, 12))
    params = wl.gen_params(spec, 9, True, "random")
    batch = wl.gen_images(4, (32, 12, 12), "normal", True, seed=1)
    x = torch.from_numpy(batch).to(DEV)
    direct_id = len(tile_configs())
    with Ensemble([spec], [params], precision="bf16", max_batch=4) as ens:
        z0, _ = logits_and_tiles(ens, x, 4)
        ens.force_tile(RAFIKI_TILE_DIRECT)
        z1, tiles = logits_and_tiles(ens, x, 4)
        assert direct_id not in tiles
        assert np.array_equal(z0.view(np.uint32), z1.view(np.uint32))
        ens.force_tile(-1)
        with pytest.raises(RafikiError):
            ens.force_tile(direct_id + 7)

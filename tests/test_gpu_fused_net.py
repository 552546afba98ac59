"""The whole-network kernel for small image CNNs (Section 5.1: every selected model
runs the batch; one workgroup per image and model runs all of a CIFAR ResNet's layers
with its activations in LDS).

The kernel sums every output in the layer-by-layer path's order, so its logits,
probabilities and labels must be bitwise those of a handle created with
RAFIKI_FUSED_NET=0 (the layer path, itself checked against the oracle in the parity
tests).  Covered: every subset of the ResNet-20 ensemble, batch sizes that put images
in every MFMA column (n = 1 .. 64) and ragged ones, both average-pool summation orders
(n * 8 >= 16384 sums the 64 positions in sequence, below that in strided partial
sums), ensembles whose members have different programs in one launch, and a model the
kernel does not take (it runs layer by layer beside the fused ones).
"""
import os

import numpy as np
import pytest
import torch

import envutil
import oracle
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def make(specs, params, max_batch, fused, autotune=True):
    return envutil.create({"RAFIKI_FUSED_NET": "1" if fused else "0", "RAFIKI_AUTOTUNE": "1" if autotune else "0"},
                          specs, params, "bf16", max_batch)


def run(ens, x, n, mask, C):
    p = torch.full((n, C), -1.0, dtype=torch.float32, device=DEV)
    lab = torch.full((n,), -7, dtype=torch.int32, device=DEV)
    ens.infer(x, n, mask, p, lab)
    torch.cuda.synchronize()
    return p.cpu().numpy(), lab.cpu().numpy()


def logits(ens, m, x, n, C):
    out = torch.full((n, C), -1.0, dtype=torch.float32, device=DEV)
    ens.model_logits(m, x, n, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def kinds(ens, x, n, mask, C):
    ens.trace(True)
    run(ens, x, n, mask, C)
    recs = ens.trace_read()
    ens.trace(False)
    return [r["kind"] for r in recs]


def compare(f, u, x, ns, masks, C, n_models):
    for n in ns:
        for mask in masks:
            pf, lf = run(f, x, n, mask, C)
            pu, lu = run(u, x, n, mask, C)
            assert np.array_equal(pf, pu) and np.array_equal(lf, lu), (n, mask)
        for m in range(n_models):
            assert np.array_equal(logits(f, m, x, n, C), logits(u, m, x, n, C)), (n, m)


def test_resnet20x3_fused_equals_layer_path():
    cfg, specs, params, batch = wl.build_config(2)
    n = cfg.n
    x = torch.from_numpy(batch).to(DEV)
    with make(specs, params, n, True) as f, make(specs, params, n, False) as u:
        compare(f, u, x, [n, 37, 1, 64, 33], range(1, 8), 10, 3)
        k = kinds(f, x, n, 0b111, 10)
        assert k.count("fused_net") == 1 and "conv_mfma" not in k, k
        assert "fused_net" not in kinds(u, x, n, 0b111, 10)
        pf, lf = run(f, x, n, 0b111, 10)
    # against the oracle's stored logits (same tie excuse as the parity tests)
    ref = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                               "oracle_logits_resnet20x3_n128.npz"))
    p_ref = oracle.combine_mean([oracle.softmax(ref[f"bf16_m{m}"]) for m in range(3)])
    srt = np.sort(p_ref, 1)
    assert not ((lf != oracle.argmax_first(p_ref)) & ((srt[:, -1] - srt[:, -2]) >= 1e-3)).any()
    assert np.abs(pf - p_ref).max() < 2e-2


def test_average_pool_orders_at_the_batch_threshold():
    """n = 2048 (2048 * 8 = 16384 (image, 8-channel) pairs) sums positions in sequence;
    n = 2047 in strided partial sums.  The fused kernel follows either."""
    spec = wl.resnet20()
    params = [wl.gen_params(spec, 31, True, "random")]
    batch = wl.gen_images(2048, spec.input_shape, "uniform", True, seed=5)
    x = torch.from_numpy(batch).to(DEV)
    with make([spec], params, 2048, True) as f, make([spec], params, 2048, False, autotune=False) as u:
        compare(f, u, x, [2048, 2047], [1], 10, 1)


def test_members_with_different_programs_in_one_launch():
    """ResNet-8 (8/16/32 wide, 40 classes: two FC channel blocks), ResNet-14 and
    ResNet-20 in one ensemble: one launch runs three different layer programs."""
    specs = [wl.resnet_cifar(1, (8, 16, 32), n_classes=40), wl.resnet_cifar(2, (16, 32, 64), n_classes=40),
             wl.resnet_cifar(3, (16, 32, 64), n_classes=40)]
    params = [wl.gen_params(s, 40 + i, True, "random") for i, s in enumerate(specs)]
    batch = wl.gen_images(70, specs[0].input_shape, "uniform", True, seed=11)
    x = torch.from_numpy(batch).to(DEV)
    with make(specs, params, 70, True) as f, make(specs, params, 70, False) as u:
        compare(f, u, x, [70, 31], [0b111, 0b101, 0b010], 40, 3)
        assert kinds(f, x, 70, 0b111, 40).count("fused_net") == 1
        pf, lf = run(f, x, 70, 0b111, 40)
    p_ref, l_ref, _ = oracle.ensemble(specs, params, batch, 0b111, act="bf16")
    srt = np.sort(p_ref, 1)
    assert not ((lf != l_ref) & ((srt[:, -1] - srt[:, -2]) >= 1e-3)).any()
    assert np.abs(pf - p_ref).max() < 2e-2


def test_model_outside_the_kernel_runs_layer_by_layer():
    """A toy CNN with a max-pool does not fit the kernel: a subset with it runs every
    model layer by layer, a subset of the ResNets alone runs fused."""
    cfg2, specs2, params2, batch = wl.build_config(2, n=16)
    toy = wl.build_config(1, n=1)[1][0]
    specs = [specs2[0], toy, specs2[1]]
    params = [params2[0], wl.gen_params(toy, 7, True, "random"), params2[1]]
    x = torch.from_numpy(batch).to(DEV)
    with make(specs, params, 16, True) as f, make(specs, params, 16, False) as u:
        compare(f, u, x, [16, 5], [0b101, 0b111, 0b010, 0b001], 10, 3)
        assert kinds(f, x, 16, 0b101, 10).count("fused_net") == 1
        k = kinds(f, x, 16, 0b111, 10)
        assert "fused_net" not in k and "conv_mfma" in k

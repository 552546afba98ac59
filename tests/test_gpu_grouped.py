"""Grouped launches of identical ensemble members (Section 5.1: a batch is served by
every selected model; models with the same layer list run each layer as one launch).

A grouped launch gives member k its own pointers on grid z = k and shares the shapes,
the tile and the K splits, so every member's logits -- and therefore the ensemble's
probabilities and labels -- must be bitwise those of the same handle with grouping
off (RAFIKI_GROUPED=0 at create, one launch per model).  The ungrouped path is itself
checked against the oracle in the parity tests; here the grouped outputs are also
checked against the oracle's labels.
"""
import os

import numpy as np
import pytest
import torch

import envutil
import oracle
import workloads as wl
from workloads import ModelSpec

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def make(specs, params, precision, max_batch, grouped):
    # the layer-by-layer path (the whole-network kernel would run the ResNets in one launch)
    return envutil.create({"RAFIKI_GROUPED": "1" if grouped else "0", "RAFIKI_FUSED_NET": "0"}, specs, params,
                          precision, max_batch)


def run(ens, x, n, mask, C):
    p = torch.full((n, C), -1.0, dtype=torch.float32, device=DEV)
    lab = torch.full((n,), -7, dtype=torch.int32, device=DEV)
    ens.infer(x, n, mask, p, lab)
    torch.cuda.synchronize()
    return p.cpu().numpy(), lab.cpu().numpy()


def launches(ens, x, n, mask, C):
    ens.trace(True)
    run(ens, x, n, mask, C)
    recs = ens.trace_read()
    ens.trace(False)
    return recs


def check_pair(specs, params, batch, precision, ns, masks, C, max_batch, group_mask=None):
    x = torch.from_numpy(batch).to(DEV)
    with make(specs, params, precision, max_batch, True) as g, make(specs, params, precision, max_batch, False) as u:
        for n in ns:
            for mask in masks:
                pg, lg = run(g, x, n, mask, C)
                pu, lu = run(u, x, n, mask, C)
                assert np.array_equal(pg, pu) and np.array_equal(lg, lu), (n, mask)
        # the grouped handle really groups: one launch per op for the selected members
        gm = (1 << len(specs)) - 1 if group_mask is None else group_mask
        rg, ru = launches(g, x, ns[0], gm, C), launches(u, x, ns[0], gm, C)
        assert len(rg) < len(ru), (len(rg), len(ru))
    return pg, lg


def test_grouped_resnet20x3_bf16():
    cfg, specs, params, batch = wl.build_config(2)
    n = cfg.n
    pg, lg = check_pair(specs, params, batch, "bf16", [n, 37, 1], range(1, 8), 10, n)
    ref = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                               "oracle_logits_resnet20x3_n128.npz"))
    p_ref = oracle.combine_mean([oracle.softmax(ref[f"bf16_m{m}"]) for m in range(3)])
    srt = np.sort(p_ref, 1)
    assert not ((lg != oracle.argmax_first(p_ref)) & ((srt[:, -1] - srt[:, -2]) >= 1e-3)).any()


def test_grouped_textcnn_x4_bf16():
    """Fused branches with the max in the GEMM epilogue (n = 512, 67) and split K (n = 5)."""
    cfg, specs, params, batch = wl.build_config(5)
    check_pair(specs, params, batch, "bf16", [cfg.n, 67, 5], [0b1111, 0b0110, 0b1011], 2, cfg.n)


def test_grouped_toy_fp32():
    cfg, specs, params, batch = wl.build_config(1)
    check_pair(specs, params, batch, "fp32", [cfg.n, 3], [0b11], 10, cfg.n)


def test_grouped_five_members_in_chunks():
    """Five identical ResNet-20s: two grouped launches per op (4 + 1 members)."""
    spec = wl.build_config(2, n=1)[1][0]
    specs = [spec] * 5
    params = [wl.gen_params(spec, 20 + i, True, "random") for i in range(5)]
    batch = wl.gen_images(24, spec.input_shape, "uniform", True, seed=9)
    check_pair(specs, params, batch, "bf16", [24, 7], [0b11111, 0b10101, 0b01111], 10, 24)


def test_mixed_ensemble_groups_only_identical_members():
    """Two ResNet-20s and a toy CNN of the same input: the ResNets group, the toy CNN
    runs on its own; a selection across both kinds runs ungrouped."""
    cfg2, specs2, params2, batch = wl.build_config(2, n=16)
    toy = wl.build_config(1, n=1)[1][0]
    toy_params = wl.gen_params(toy, 7, True, "random")
    specs = [specs2[0], specs2[1], toy]
    params = [params2[0], params2[1], toy_params]
    check_pair(specs, params, batch, "bf16", [16, 5], [0b011, 0b111, 0b101, 0b100], 10, 16, group_mask=0b011)
    x = torch.from_numpy(batch).to(DEV)
    with make(specs, params, "bf16", 16, True) as g, make(specs, params, "bf16", 16, False) as u:
        assert len(launches(g, x, 16, 0b111, 10)) == len(launches(u, x, 16, 0b111, 10))

"""Schedules of the selected models' forward passes (rafiki_ensemble_get/set_schedule).

A schedule only orders the same launches across the model streams (all concurrent, or
one model alone on a lane while the others run one after another on a second lane), so
every schedule must give bit-identical probabilities and labels; the one chosen by
timing on the first call must be a valid candidate.
"""
import os

import numpy as np
import pytest
import torch

import envutil
import workloads as wl
from paper_1804_06087_amd import Ensemble, RafikiError, RAFIKI_ERR_INVALID

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _ungrouped(specs, params, max_batch):
    """Schedules order the models' own streams, so identical members (which otherwise
    run as grouped launches on one stream, or the ResNets as one whole-network launch)
    are created on the layer-by-layer path with grouping off."""
    return envutil.create(envutil.LAYER_PATH, specs, params, "bf16", max_batch)


def _infer(ens, x, n, mask, C, vote=False):
    p = torch.empty((n, C), dtype=torch.float32, device=DEV)
    lab = torch.empty((n,), dtype=torch.int32, device=DEV)
    (ens.infer_vote if vote else ens.infer)(x, n, mask, p, lab)
    torch.cuda.synchronize()
    return p.cpu().numpy(), lab.cpu().numpy()


@pytest.mark.parametrize("cid,n,mask", [(2, 37, 0b111), (5, 40, 0b1111), (5, 40, 0b1011)])
def test_every_schedule_gives_the_same_bits(cid, n, mask):
    cfg, specs, params, batch = wl.build_config(cid, n=n)
    C = specs[0].n_classes
    x = torch.from_numpy(batch).to(DEV)
    with _ungrouped(specs, params, n) as ens:
        p0, l0 = _infer(ens, x, n, mask, C)
        chosen, asc = ens.get_schedule(n, mask)
        members = [m for m in range(len(specs)) if (mask >> m) & 1]
        assert chosen == -1 or chosen in members
        assert asc in (0, 1)
        v0 = _infer(ens, x, n, mask, C, vote=True)
        for solo, asc in [(-1, 0)] + [(m, a) for m in members for a in (0, 1)]:
            ens.set_schedule(n, mask, solo, asc)
            assert ens.get_schedule(n, mask) == (solo, asc)
            for _ in range(2):
                p, lab = _infer(ens, x, n, mask, C)
                assert np.array_equal(p, p0), f"schedule {solo}/{asc}: probabilities differ"
                assert np.array_equal(lab, l0), f"schedule {solo}/{asc}: labels differ"
            v, lv = _infer(ens, x, n, mask, C, vote=True)
            assert np.array_equal(v, v0[0]) and np.array_equal(lv, v0[1])


def test_schedule_arguments():
    cfg, specs, params, batch = wl.build_config(2, n=8)
    with _ungrouped(specs, params, 8) as ens:
        with pytest.raises(RafikiError) as e:
            ens.get_schedule(8, 0b111)                 # nothing chosen yet
        assert e.value.code == RAFIKI_ERR_INVALID
        with pytest.raises(RafikiError):
            ens.set_schedule(8, 0b011, 2)              # model 2 is not in the subset
        with pytest.raises(RafikiError):
            ens.set_schedule(9, 0b111, -1)             # beyond max_batch
        with pytest.raises(RafikiError):
            ens.set_schedule(8, 0b1000, -1)            # no such model
        ens.set_schedule(8, 0b111, 1, 1)
        assert ens.get_schedule(8, 0b111) == (1, 1)


def test_lean_tiles_give_the_same_bits():
    """The tile policy of a schedule (rafiki_ensemble_get/set_schedule_tiles): with the
    lean tiles the layers of maps up to 14 x 14 run on 8-wave tiles of at least 128 x 128
    with K tiles of 64 and at most 64 KB of LDS ring, with policy 2 also the solo model's
    direct-conv layers on GEMM tiles, and the results are bit-identical to the fastest
    tiles alone; set_schedule resets the policy."""
    from paper_1804_06087_amd.binding import tile_configs
    n, mask = 8, 0b111
    cfg, specs, params, batch = wl.build_config(3, n=n)   # ResNet-50, VGG-16, ResNet-101
    C = specs[0].n_classes
    x = torch.from_numpy(batch).to(DEV)
    tiles = tile_configs()
    lean_ids = {i for i, t in enumerate(tiles)
                if t["waves"] == 8 and t["bm"] * t["bn"] >= 128 * 128 and t["bk"] == 64
                and t["stages"] * (t["bm"] + t["bn"]) * t["bk"] * 2 <= 65536}
    assert lean_ids
    with Ensemble(specs, params, precision="bf16", max_batch=n) as ens:
        with pytest.raises(RafikiError):
            ens.get_schedule_tiles(n, mask)           # nothing chosen yet
        p0, l0 = _infer(ens, x, n, mask, C)
        assert ens.get_schedule_tiles(n, mask) in (0, 1, 2)
        with pytest.raises(RafikiError):
            ens.set_schedule_tiles(n, mask, 3)
        with pytest.raises(RafikiError):
            ens.set_schedule_tiles(n, 0b011, 1)       # no schedule kept for this subset
        ens.set_schedule(n, mask, 2, 0)                # ResNet-101 alone on a lane
        for lean in (1, 0, 2, 1):
            ens.set_schedule_tiles(n, mask, lean)
            assert ens.get_schedule_tiles(n, mask) == lean
            for _ in range(2):
                p, lab = _infer(ens, x, n, mask, C)
                assert np.array_equal(p, p0), f"lean {lean}: probabilities differ"
                assert np.array_equal(lab, l0), f"lean {lean}: labels differ"
            ens.trace(True, concurrent=True)
            _infer(ens, x, n, mask, C)
            recs = ens.trace_read()
            ens.trace(False)
            small = [r for r in recs if r["kind"] == "conv_mfma" and r["splits"] == 1 and r["tile_cfg"] < len(tiles)
                     and r["flops"] > 0]
            used = {r["tile_cfg"] for r in small}
            if lean:
                assert used & lean_ids, used
            direct_r101 = [r for r in recs if r["kind"] == "conv_mfma" and r["model"] == 2 and r["tile_cfg"] == len(tiles)]
            if lean == 2:
                assert not direct_r101       # the solo model's direct-conv layers on GEMM tiles
        solo, asc = ens.get_schedule(n, mask)
        ens.set_schedule(n, mask, solo, asc)
        assert ens.get_schedule_tiles(n, mask) == 0

"""Graph replay of the forward passes (rafiki_ensemble_use_graphs / _graph_stats).

With graphs on (they are opt-in), once a batch size is tuned, infer captures the forward passes of (n, mask) into a HIP
graph and replays it, with staging and the combine launched around it.  The replayed
results must equal the eager launches bit for bit: every replay is checked against the
eager result of the same input, with eager work, other inputs and synchronisations
between replays (a graph that read a stale staged input, or skipped a node, would
differ).  One case is also checked against the oracle.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import envutil
import workloads as wl
from paper_1804_06087_amd import Ensemble

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _infer(ens, x, n, mask, C, vote=False):
    p = torch.empty((n, C), dtype=torch.float32, device=DEV)
    lab = torch.empty((n,), dtype=torch.int32, device=DEV)
    (ens.infer_vote if vote else ens.infer)(x, n, mask, p, lab)
    torch.cuda.synchronize()
    return p.cpu().numpy(), lab.cpu().numpy()


def _replay_matches_eager(ens, inputs, n, masks, C, vote=False):
    ens.use_graphs(False)
    eager = {(i, m): _infer(ens, x, n, m, C, vote) for i, x in enumerate(inputs) for m in masks}
    ens.use_graphs(True)
    g0, r0, f0 = ens.graph_stats()
    assert g0 == 0 and f0 == 0
    for rep in range(3):
        for i, x in enumerate(inputs):
            for m in masks:
                p, lab = _infer(ens, x, n, m, C, vote)
                pe, le = eager[(i, m)]
                assert np.array_equal(p, pe), f"replay {rep} input {i} mask {m}: probabilities differ"
                assert np.array_equal(lab, le), f"replay {rep} input {i} mask {m}: labels differ"
        # eager work on the same handle between replays
        ens.trace(True)
        _infer(ens, inputs[0], n, masks[0], C, vote)
        ens.trace(False)
    g, r, f = ens.graph_stats()
    assert f == 0, "a graph capture failed"
    assert g == len(masks)
    assert r - r0 == 3 * len(inputs) * len(masks)


def test_graph_replay_resnet20_ragged_and_full():
    cfg, specs, params, batch = wl.build_config(2, n=128)
    C = 10
    x_full = torch.from_numpy(batch).to(DEV)
    x_alt = torch.from_numpy(np.ascontiguousarray(batch[::-1])).to(DEV)
    with Ensemble(specs, params, precision="bf16", max_batch=128) as ens:
        for n in (37, 128):
            _infer(ens, x_full, n, 0b111, C)          # tunes n (eager)
            _replay_matches_eager(ens, [x_full[:n], x_alt[:n]], n, [0b111, 0b010, 0b101], C)
            _replay_matches_eager(ens, [x_full[:n]], n, [0b111, 0b011], C, vote=True)


def test_graph_replay_against_oracle():
    cfg, specs, params, batch = wl.build_config(2, n=9)
    C = 10
    x = torch.from_numpy(batch).to(DEV)
    zb = [oracle.run_model(s, p, batch, act="bf16") for s, p in zip(specs, params)]
    with Ensemble(specs, params, precision="bf16", max_batch=16) as ens:
        ens.use_graphs(True)
        _infer(ens, x, 9, 0b111, C)                    # eager, tunes n = 9
        for _ in range(2):
            p, lab = _infer(ens, x, 9, 0b110, C)       # captured, then replayed
            p_ref, _, _ = oracle.ensemble(specs, params, batch, 0b110, logits=zb)
            assert np.allclose(p.sum(1), 1.0, atol=1e-5)
            assert np.abs(p - p_ref).max() <= 2e-2
            srt = np.sort(p_ref, 1)
            sure = (srt[:, -1] - srt[:, -2]) >= 1e-3
            assert np.array_equal(lab[sure], oracle.argmax_first(p_ref)[sure])
        assert ens.graph_stats()[1] == 2


def test_graph_replay_tokens():
    cfg, specs, params, batch = wl.build_config(5, n=40)
    C = 2
    specs, params = specs[:2], params[:2]
    x = torch.from_numpy(batch).to(DEV)
    x_alt = torch.from_numpy(np.ascontiguousarray(batch[::-1])).to(DEV)
    with Ensemble(specs, params, precision="bf16", max_batch=40) as ens:
        _infer(ens, x, 40, 0b11, C)
        _replay_matches_eager(ens, [x, x_alt], 40, [0b11, 0b01], C)
        _infer(ens, x, 23, 0b11, C)                    # ragged batch size: tuned eagerly first
        _replay_matches_eager(ens, [x[:23], x_alt[:23]], 23, [0b11], C)
        # n = 40 and 23: the fused branch GEMM takes the max over time in its epilogue
        # (slots reset by the finishing kernel); n = 5 splits K and stores the rows
        _infer(ens, x, 5, 0b11, C)
        _replay_matches_eager(ens, [x[:5], x_alt[:5]], 5, [0b11, 0b10], C)


def test_graph_dropped_by_force_tile():
    cfg, specs, params, batch = wl.build_config(2, n=16)
    C = 10
    x = torch.from_numpy(batch).to(DEV)
    with envutil.create({"RAFIKI_FUSED_NET": "0"}, specs, params, "bf16", 16) as ens:   # tiles: the layer path
        ens.use_graphs(True)
        base = _infer(ens, x, 16, 0b111, C)
        p, lab = _infer(ens, x, 16, 0b111, C)          # captured
        assert ens.graph_stats()[0] == 1
        ens.force_tile(8)                              # 64x64 tiles: same sums, new graph
        assert ens.graph_stats()[0] == 0
        p2, lab2 = _infer(ens, x, 16, 0b111, C)
        ens.force_tile(-1)
        assert np.array_equal(p, base[0]) and np.array_equal(p2, base[0])
        assert np.array_equal(lab2, base[1])
        assert ens.graph_stats()[2] == 0


@pytest.mark.parametrize("solo,asc", [(-1, 0), (0, 0), (2, 1)])
def test_graph_replay_under_each_schedule(solo, asc):
    """A graph captured with a two-lane schedule (a model waiting on another's done
    event) replays the same bits as the eager launches."""
    cfg, specs, params, batch = wl.build_config(2, n=24)
    C = 10
    x = torch.from_numpy(batch).to(DEV)
    # schedules order the models' own streams (no grouped or whole-network launches)
    with envutil.create(envutil.LAYER_PATH, specs, params, "bf16", 24) as ens:
        _infer(ens, x, 24, 0b111, C)                   # tunes n = 24
        ens.set_schedule(24, 0b111, solo, asc)
        ens.use_graphs(False)
        base = _infer(ens, x, 24, 0b111, C)
        ens.use_graphs(True)
        for _ in range(3):
            p, lab = _infer(ens, x, 24, 0b111, C)
            assert np.array_equal(p, base[0]) and np.array_equal(lab, base[1])
        g, r, f = ens.graph_stats()
        assert g == 1 and r == 3 and f == 0

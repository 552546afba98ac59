"""Paired layers of two different models (Section 5.1: the selected models all run the
batch): ResNet-50's ops align with ops of ResNet-101 of the same launch shapes, and a
paired schedule runs each aligned pair as one launch with a member per model.

Every member's outputs are those of its own launch, so probabilities and labels must
be bitwise those of the unpaired schedules, for the three-model ensemble (VGG-16 on the
second lane) and for the pair alone; the traced launches must show the pairing (one
conv launch fewer per aligned conv).
"""
import numpy as np
import pytest
import torch

import workloads as wl
from paper_1804_06087_amd import Ensemble, RafikiError, RAFIKI_ERR_INVALID

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
R50, VGG, R101 = 0, 1, 2


@pytest.fixture(scope="module")
def c3():
    cfg, specs, params, batch = wl.build_config(3, n=16)
    assert [s.name for s in specs] == ["resnet50", "vgg16", "resnet101"]
    ens = Ensemble(specs, params, precision="bf16", max_batch=16)
    yield ens, torch.from_numpy(batch).to(DEV), specs
    ens.close()


def _infer(ens, x, n, mask):
    p = torch.full((n, 1000), -1.0, dtype=torch.float32, device=DEV)
    lab = torch.full((n,), -7, dtype=torch.int32, device=DEV)
    ens.infer(x, n, mask, p, lab)
    torch.cuda.synchronize()
    return p.cpu().numpy(), lab.cpu().numpy()


def _conv_launches(ens, x, n, mask):
    ens.trace(True, concurrent=True)
    _infer(ens, x, n, mask)
    recs = ens.trace_read()
    ens.trace(False)
    return sum(r["kind"] == "conv_mfma" for r in recs)


def test_resnet50_aligns_within_resnet101(c3):
    ens, x, specs = c3
    aligned = ens.pairing(R50, R101)
    n_r50 = sum(1 for L in specs[R50].layers)   # every ResNet-50 layer has a ResNet-101 twin
    assert aligned >= n_r50 - 2, (aligned, n_r50)
    assert ens.pairing(R50, VGG) == 0 and ens.pairing(VGG, R101) == 0


@pytest.mark.parametrize("n,mask", [(16, 0b111), (4, 0b111), (16, 0b101), (3, 0b101)])
def test_paired_schedule_gives_the_same_bits(c3, n, mask):
    ens, x, specs = c3
    ens.set_schedule(n, mask, -1, 0)                  # every model on its own lane
    p0, l0 = _infer(ens, x, n, mask)
    c0 = _conv_launches(ens, x, n, mask)
    ens.set_schedule_pair(n, mask, R50, R101)
    assert ens.get_schedule_pair(n, mask) == (R50, R101)
    for _ in range(2):
        p, lab = _infer(ens, x, n, mask)
        assert np.array_equal(p, p0) and np.array_equal(lab, l0)
    c1 = _conv_launches(ens, x, n, mask)
    assert c1 < c0 - 40, (c0, c1)
    ens.set_schedule_pair(n, mask, -1, -1)
    assert ens.get_schedule_pair(n, mask) == (-1, -1)


def test_timed_schedule_is_a_candidate(c3):
    ens, x, specs = c3
    _infer(ens, x, 8, 0b111)                          # times the candidates for (8, all)
    solo, asc = ens.get_schedule(8, 0b111)
    pa, pb = ens.get_schedule_pair(8, 0b111)
    assert (pa, pb) in ((-1, -1), (R50, R101))
    assert solo in (-1, R50, VGG, R101)


def test_schedule_pair_argument_errors(c3):
    ens, x, specs = c3
    for a, b in ((R101, R50), (R50, VGG), (R50, 7)):
        with pytest.raises(RafikiError) as ei:
            ens.set_schedule_pair(16, 0b111, a, b)
        assert ei.value.code == RAFIKI_ERR_INVALID
    with pytest.raises(RafikiError):
        ens.set_schedule_pair(16, 0b011, R50, R101)   # R101 not in the subset

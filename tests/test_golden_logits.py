"""The stored oracle logits the GPU parity tests read are the oracle's.

``tests/golden/oracle_logits_*.npz`` hold ``oracle.run_model``'s per-model logits of
the configured request batches (written by ``tests/golden/make_oracle_logits.py``).
Sample rows of each file -- the first and the last, and one in between -- are
recomputed here from the oracle on the same seeded parameters and inputs, so a file
that drifted from the oracle or from the workload generator fails on the CPU.
"""
import os

import numpy as np
import pytest

import oracle
import workloads as wl

GOLD = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
CASES = [
    ("oracle_logits_resnet20x3_n128.npz", 2, 128, (0, 77, 127)),
    ("oracle_logits_textcnn_x4_n512.npz", 5, 512, (0, 300, 511)),
    ("oracle_logits_r50_vgg16_r101_n256.npz", 4, 256, (0, 255)),
]


@pytest.mark.parametrize("fname,cid,n,rows", CASES)
def test_stored_logits_are_the_oracles(fname, cid, n, rows):
    d = np.load(os.path.join(GOLD, fname))
    cfg, specs, params, batch = wl.build_config(cid)
    assert batch.shape[0] == n
    rows = list(rows)
    for m, (s, p) in enumerate(zip(specs, params)):
        for mode, act in (("exact", None), ("bf16", "bf16")):
            z = d[f"{mode}_m{m}"]
            assert z.shape == (n, s.n_classes) and z.dtype == np.float64
            assert np.isfinite(z).all()
            ref = oracle.run_model(s, p, batch[rows], act=act, chunk=2)
            scale = np.abs(ref).max(1, keepdims=True)
            assert (np.abs(z[rows] - ref) <= 1e-9 * scale).all(), (fname, m, mode)

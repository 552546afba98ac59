"""Majority-vote combine (Section 5.2) through the C ABI.

The vote is integer work on top of each model's logits, so it is checked in two parts:
* the combine itself is exact: the GPU's vote fractions and labels equal the oracle's
  ``combine_vote`` applied to the GPU's own per-model fp32 logits (same precision on
  both sides for the argmax decisions);
* each model's prediction (first-index argmax of its logits) equals the oracle's,
  except on rows whose oracle top-2 logit gap lies within twice the logit tolerance
  (fp32: 1e-4, bf16: 2e-2, row-normwise), where rounding may legitimately flip it.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from workloads import Layer, ModelSpec, FC
from paper_1804_06087_amd import Ensemble, RafikiError, RAFIKI_ERR_INVALID

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
CANARY = 7777.0


def run_vote(ens, batch_np, n, mask, C):
    x = torch.from_numpy(np.ascontiguousarray(batch_np[:n])).to(DEV)
    votes = torch.full((n * C + 64,), CANARY, dtype=torch.float32, device=DEV)
    labels = torch.full((n + 16,), -7, dtype=torch.int32, device=DEV)
    ens.infer_vote(x, n, mask, votes, labels)
    torch.cuda.synchronize()
    v = votes.cpu().numpy()
    lab = labels.cpu().numpy()
    assert (v[n * C:] == CANARY).all(), "write past out_votes"
    assert (lab[n:] == -7).all(), "write past out_labels"
    return v[:n * C].reshape(n, C), lab[:n]


def run_logits(ens, batch_np, n, m, C):
    x = torch.from_numpy(np.ascontiguousarray(batch_np[:n])).to(DEV)
    out = torch.empty((n, C), dtype=torch.float32, device=DEV)
    ens.model_logits(m, x, n, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def check_combine_exact(v, lab, z_sel):
    v_ref, l_ref = oracle.combine_vote([z.astype(np.float64) for z in z_sel])
    assert np.array_equal(lab, l_ref), f"labels differ at rows {np.nonzero(lab != l_ref)[0]}"
    assert np.abs(v - v_ref).max() <= 1e-6
    assert np.allclose(v.sum(1), 1.0, atol=1e-5)


def check_predictions(z_gpu, z_ref, tol):
    """Model prediction parity, excusing rows whose top-2 gap is within 2 * tol * max|z|."""
    z_ref = np.asarray(z_ref, np.float64)
    srt = np.sort(z_ref, 1)
    gap = (srt[:, -1] - srt[:, -2]) / np.maximum(np.abs(z_ref).max(1), 1e-30)
    diff = oracle.argmax_first(z_gpu.astype(np.float64)) != oracle.argmax_first(z_ref)
    bad = diff & (gap > 2 * tol)
    assert not bad.any(), f"prediction flips outside the rounding band at rows {np.nonzero(bad)[0]}"
    return diff.mean()


def test_vote_c1_fp32_all_masks():
    cfg, specs, params, batch = wl.build_config(1)
    n, C = cfg.n, 10
    with Ensemble(specs, params, precision="fp32", max_batch=8) as ens:
        zg = [run_logits(ens, batch, n, m, C) for m in range(2)]
        zo = [oracle.run_model(s, p, batch) for s, p in zip(specs, params)]
        for m in range(2):
            check_predictions(zg[m], zo[m], 1e-4)
        for mask in (1, 2, 3):
            v, lab = run_vote(ens, batch, n, mask, C)
            sel = [m for m in range(2) if (mask >> m) & 1]
            check_combine_exact(v, lab, [zg[m] for m in sel])
            if all((oracle.argmax_first(zg[m]) == oracle.argmax_first(zo[m])).all() for m in sel):
                _, l_o, _ = oracle.ensemble_vote(specs, params, batch, mask, logits=zo)
                assert np.array_equal(lab, l_o)


def test_vote_c2_bf16_all_masks_ragged():
    cfg, specs, params, batch = wl.build_config(2, n=37)
    n, C = 37, 10
    zb = [oracle.run_model(s, p, batch, act="bf16") for s, p in zip(specs, params)]
    with Ensemble(specs, params, precision="bf16", max_batch=48) as ens:
        zg = [run_logits(ens, batch, n, m, C) for m in range(3)]
        for m in range(3):
            check_predictions(zg[m], zb[m], 2e-2)
        for mask in range(1, 8):
            v, lab = run_vote(ens, batch, n, mask, C)
            check_combine_exact(v, lab, [zg[m] for m in range(3) if (mask >> m) & 1])
            v2, lab2 = run_vote(ens, batch, n, mask, C)
            assert np.array_equal(v, v2) and np.array_equal(lab, lab2), "not deterministic"
        # a single selected model's vote is its own prediction
        v, lab = run_vote(ens, batch, n, 0b010, C)
        assert np.array_equal(lab, oracle.argmax_first(zg[1].astype(np.float64)))


def _fc_model(n_classes, in_shape):
    c, h, w = in_shape
    return ModelSpec("fc_probe", [Layer(op=FC, input=-1, c_in=c * h * w, c_out=n_classes, bias=True)],
                     n_classes, in_shape)


def test_vote_priority_ties():
    """Models 0 = 1 and 2 = 3 (identical weights): selecting all four ties 2-2 wherever
    the pairs disagree, and the tie goes to model 0's class; {1, 2, 3} is a 2-1
    majority for the second pair's class."""
    shape, C, n = (3, 4, 4), 9, 40
    spec = _fc_model(C, shape)
    pa, pb = wl.gen_params(spec, 21, False, "random"), wl.gen_params(spec, 22, False, "random")
    batch = wl.gen_images(n, shape, "normal", False, seed=4)
    with Ensemble([spec] * 4, [pa, pa, pb, pb], precision="fp32", max_batch=n) as ens:
        za, zb_ = run_logits(ens, batch, n, 0, C), run_logits(ens, batch, n, 2, C)
        pred_a = oracle.argmax_first(za.astype(np.float64))
        pred_b = oracle.argmax_first(zb_.astype(np.float64))
        assert (pred_a != pred_b).sum() >= 10, "the two weight sets should disagree often"
        _, lab = run_vote(ens, batch, n, 0b1111, C)
        assert np.array_equal(lab, pred_a)
        _, lab = run_vote(ens, batch, n, 0b1110, C)
        assert np.array_equal(lab, pred_b)
        v, lab = run_vote(ens, batch, n, 0b1100, C)
        assert np.array_equal(lab, pred_b) and set(np.unique(v)) <= {0.0, 1.0}
        v, lab = run_vote(ens, batch, n, 0b0110, C)
        assert np.array_equal(lab, pred_a)                  # model 1 outranks model 2
        assert np.allclose(v[pred_a != pred_b].max(1), 0.5)


def test_vote_32_models_full_mask():
    """The largest ensemble: 32 models, mask 0xFFFFFFFF, and a few sparse masks."""
    shape, C, n = (3, 4, 4), 7, 33
    spec = _fc_model(C, shape)
    params = [wl.gen_params(spec, 100 + m, False, "random") for m in range(32)]
    batch = wl.gen_images(n, shape, "normal", False, seed=8)
    zo = [oracle.run_model(spec, p, batch) for p in params]
    with Ensemble([spec] * 32, params, precision="fp32", max_batch=n) as ens:
        zg = [run_logits(ens, batch, n, m, C) for m in range(32)]
        for m in range(32):
            check_predictions(zg[m], zo[m], 1e-4)
        for mask in (0xFFFFFFFF, 0x80000001, 0x55555555, 0x80000000):
            v, lab = run_vote(ens, batch, n, mask, C)
            check_combine_exact(v, lab, [zg[m] for m in range(32) if (mask >> m) & 1])


def test_vote_c3_full_batch(c3_vote_ens):
    """Every row of the batch of 64: each model's prediction against the oracle's
    (stored fp64 logits, both modes), then the exact vote."""
    ens, specs, params, batch, ref = c3_vote_ens
    n, C = 64, 1000
    zg = [run_logits(ens, batch, n, m, C) for m in range(3)]
    for m in range(3):
        for mode in ("bf16", "exact"):
            check_predictions(zg[m], ref[f"{mode}_m{m}"][:n], 2e-2)
    for mask in (0b111, 0b101, 0b011):
        v, lab = run_vote(ens, batch, n, mask, C)
        check_combine_exact(v, lab, [zg[m] for m in range(3) if (mask >> m) & 1])


@pytest.fixture(scope="module")
def c3_vote_ens():
    cfg, specs, params, batch = wl.build_config(3)
    ref = np.load(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                               "oracle_logits_r50_vgg16_r101_n256.npz"))
    ens = Ensemble(specs, params, precision="bf16", max_batch=64)
    yield ens, specs, params, batch, ref
    ens.close()


def test_vote_argument_errors():
    cfg, specs, params, batch = wl.build_config(1)
    with Ensemble(specs, params, precision="fp32", max_batch=8) as ens:
        x = torch.from_numpy(batch).to(DEV)
        votes = torch.empty((16, 10), device=DEV)
        labels = torch.empty((16,), dtype=torch.int32, device=DEV)
        for n, mask in ((9, 1), (0, 1), (4, 0), (4, 0b100)):
            with pytest.raises(RafikiError) as ei:
                ens.infer_vote(x, n, mask, votes, labels)
            assert ei.value.code == RAFIKI_ERR_INVALID

"""Pins of the fp64 oracle against facts fixed outside it: scalar brute force, an
independent library (torch CPU float64), closed forms, invariants, published
parameter and MAC counts, and a hand-computed combine example."""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import brute
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
rng = np.random.default_rng(1234)


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


# ---------------------------------------------------------------- conv2d
@pytest.mark.parametrize("stride,pad,k", [(1, 0, 3), (1, 1, 3), (2, 1, 3), (2, 0, 1), (1, 0, 1), (2, 3, 7), (2, 1, 2)])
def test_conv2d_brute_force(stride, pad, k):
    x = rng.standard_normal((2, 3, 7, 6))
    w = rng.standard_normal((4, 3, k, k))
    b = rng.standard_normal(4)
    got = oracle.conv2d(x, w, stride, pad, b)
    ref = np.array(brute.conv2d(x.tolist(), w.tolist(), stride, pad, b.tolist()))
    assert got.shape == ref.shape
    assert np.abs(got - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max())


@pytest.mark.parametrize("stride,pad,k,c", [(1, 1, 3, 16), (2, 1, 3, 8), (2, 3, 7, 3), (2, 0, 1, 32)])
def test_conv2d_torch_fp64(stride, pad, k, c):
    x = rng.standard_normal((3, c, 13, 11))
    w = rng.standard_normal((5, c, k, k))
    got = oracle.conv2d(x, w, stride, pad)
    ref = F.conv2d(_t(x), _t(w), stride=stride, padding=pad).numpy()
    assert np.abs(got - ref).max() <= 1e-12 * np.abs(ref).max()


def test_conv1x1_is_per_pixel_matmul():
    x = rng.standard_normal((2, 6, 5, 4))
    w = rng.standard_normal((7, 6, 1, 1))
    got = oracle.conv2d(x, w, 1, 0)
    ref = np.einsum("nchw,oc->nohw", x, w[:, :, 0, 0])
    assert np.allclose(got, ref, rtol=0, atol=1e-12)


def test_identity_kernel():
    x = rng.standard_normal((1, 3, 6, 5))
    w = np.zeros((3, 3, 3, 3))
    for c in range(3):
        w[c, c, 1, 1] = 1.0
    assert np.array_equal(oracle.conv2d(x, w, 1, 1), x)


def _shift_pin_holds(conv):
    """Single tap at (0, 0) with pad 1 must give out[y, x] = in[y-1, x-1] (zero-filled):
    this fixes cross-correlation against true convolution."""
    x = rng.standard_normal((1, 1, 5, 5))
    w = np.zeros((1, 1, 3, 3))
    w[0, 0, 0, 0] = 1.0
    got = conv(x, w, 1, 1)
    want = np.zeros_like(x)
    want[0, 0, 1:, 1:] = x[0, 0, :-1, :-1]
    return np.array_equal(got, want)


def test_shift_kernel_fixes_orientation():
    assert _shift_pin_holds(oracle.conv2d)


def test_planted_flip_is_caught():
    """A planted mistake (true convolution, i.e. flipped kernel) fails the shift pin."""
    def flipped(x, w, s, p):
        return oracle.conv2d(x, w[:, :, ::-1, ::-1], s, p)
    assert not _shift_pin_holds(flipped)


def test_padding_tap_counts():
    c_in, val = 4, 0.5
    x = np.full((1, c_in, 5, 6), val)
    w = np.ones((1, c_in, 3, 3))
    y = oracle.conv2d(x, w, 1, 1)[0, 0]
    assert y[2, 2] == c_in * 9 * val
    assert y[0, 2] == c_in * 6 * val and y[2, 0] == c_in * 6 * val
    assert y[0, 0] == c_in * 4 * val and y[-1, -1] == c_in * 4 * val


# ---------------------------------------------------------------- BN / pools / FC
def test_bn_identity_stats():
    x = rng.standard_normal((2, 5, 3, 3))
    y = oracle.batchnorm(x, np.ones(5), np.zeros(5), np.zeros(5), np.ones(5), 1e-5)
    assert np.allclose(y, x / math.sqrt(1 + 1e-5), rtol=1e-15, atol=0)


def test_bn_matches_torch():
    x = rng.standard_normal((2, 5, 3, 3))
    g, b, m, v = rng.standard_normal(5), rng.standard_normal(5), rng.standard_normal(5), rng.uniform(0.5, 1.5, 5)
    ref = F.batch_norm(_t(x), _t(m), _t(v), _t(g), _t(b), training=False, eps=1e-5).numpy()
    assert np.abs(oracle.batchnorm(x, g, b, m, v, 1e-5) - ref).max() < 1e-13


def test_maxpool_ramp_and_torch():
    x = np.arange(2 * 3 * 6 * 6, dtype=np.float64).reshape(2, 3, 6, 6)
    y = oracle.maxpool2d(x, 2, 2, 0)
    assert np.array_equal(y, x[:, :, 1::2, 1::2])        # a ramp's window max is its last cell
    x = rng.standard_normal((2, 4, 9, 7))
    for k, s, p in ((3, 2, 1), (2, 2, 0), (3, 1, 1)):
        ref = F.max_pool2d(_t(x), k, s, p).numpy()
        assert np.array_equal(oracle.maxpool2d(x, k, s, p), ref)
        assert np.array_equal(np.array(brute.maxpool2d(x.tolist(), k, s, p)), ref)


def test_maxpool_negative_inputs_see_minus_inf_padding():
    x = -np.ones((1, 1, 3, 3)) - np.arange(9.0).reshape(1, 1, 3, 3)
    y = oracle.maxpool2d(x, 3, 2, 1)
    assert y[0, 0, 0, 0] == -1.0                          # padding never wins


def test_gap_constant_and_mean():
    x = np.full((2, 3, 4, 5), 2.5)
    assert np.array_equal(oracle.global_avgpool(x), np.full((2, 3), 2.5))
    x = rng.standard_normal((2, 3, 4, 5))
    assert np.allclose(oracle.global_avgpool(x), F.adaptive_avg_pool2d(_t(x), 1).numpy()[:, :, 0, 0], atol=1e-15)


def test_fc_one_hot_and_brute():
    w = rng.standard_normal((5, 8))
    b = rng.standard_normal(5)
    x = np.zeros((1, 8)); x[0, 3] = 1.0
    assert np.array_equal(oracle.fc(x, w, b)[0], w[:, 3] + b)
    x = rng.standard_normal((3, 8))
    assert np.allclose(oracle.fc(x, w, b), np.array(brute.fc(x.tolist(), w.tolist(), b.tolist())), atol=1e-13)


def test_flatten_order_is_chw():
    """One-hot at (c, h, w) of a [C, H, W] input selects FC column c*H*W + h*W + w."""
    C, H, W = 3, 2, 4
    wt = rng.standard_normal((6, C * H * W))
    for (c, h, w_) in ((0, 0, 1), (2, 1, 3), (1, 0, 0)):
        x = np.zeros((1, C, H, W)); x[0, c, h, w_] = 1.0
        assert np.array_equal(oracle.fc(x, wt)[0], wt[:, c * H * W + h * W + w_])


def test_conv1d_maxtime_brute_and_torch():
    e = rng.standard_normal((2, 9, 4))
    w = rng.standard_normal((3, 4, 3))
    b = rng.standard_normal(3)
    got = oracle.conv1d_maxtime(e, w, b, True)
    ref = np.array(brute.conv1d_maxtime(e.tolist(), w.tolist(), b.tolist(), True))
    assert np.allclose(got, ref, atol=1e-13)
    y = F.relu(F.conv1d(_t(e).transpose(1, 2), _t(w), _t(b))).amax(dim=2).numpy()
    assert np.allclose(got, y, atol=1e-13)


def test_embedding_gather():
    table = rng.standard_normal((10, 4))
    tok = np.array([[3, 0, 9]])
    assert np.array_equal(oracle.embedding(tok, table)[0], table[[3, 0, 9]])


# ---------------------------------------------------------------- softmax / combine
def test_softmax_invariants():
    z = rng.standard_normal((5, 7)) * 30
    p = oracle.softmax(z)
    assert np.allclose(p.sum(1), 1.0, atol=1e-15)
    assert np.allclose(oracle.softmax(z + 123.0), p, atol=1e-15)
    assert np.allclose(p, torch.softmax(_t(z), 1).numpy(), atol=1e-15)
    for row in z[:2]:
        assert np.allclose(oracle.softmax(row[None])[0], brute.softmax_row(row.tolist()), atol=1e-15)
    d = rng.standard_normal(4)
    two = oracle.softmax(np.stack([d, np.zeros(4)], 1))
    assert np.allclose(two[:, 0], 1.0 / (1.0 + np.exp(-d)), atol=1e-15)


def test_combine_golden_example():
    g = json.load(open(os.path.join(GOLDEN, "combine_2x3.json")))
    logits = np.array(g["logits"])                       # [model, row, class]
    ints = np.array(g["logits_are_log_of"], dtype=np.float64)
    assert np.allclose(np.exp(logits), ints, rtol=1e-15)
    p = oracle.combine_mean([oracle.softmax(logits[0]), oracle.softmax(logits[1])])
    assert np.allclose(p, g["expected_probs"], atol=1e-15)
    assert oracle.argmax_first(p).tolist() == g["expected_labels"]


def test_argmax_ties_lowest_index():
    p = np.array([[0.2, 0.4, 0.4], [1 / 3, 1 / 3, 1 / 3], [0.0, 0.0, 1.0]])
    assert oracle.argmax_first(p).tolist() == [1, 0, 2]


class _Z:
    """Stand-in model whose 'forward pass' returns fixed logits (exercises only the combine)."""


def _fake_ensemble(zs, mask):
    return oracle.ensemble([None] * len(zs), [None] * len(zs), np.zeros((zs[0].shape[0], 1)), mask, logits=zs)


def test_ensemble_invariants():
    zs = [rng.standard_normal((6, 5)) * 3 for _ in range(3)]
    for m in range(3):                                   # one-model mask == that model
        p, lab, _ = _fake_ensemble(zs, 1 << m)
        assert np.allclose(p, oracle.softmax(zs[m]), atol=1e-15)
        assert np.array_equal(lab, np.argmax(zs[m], 1))
    p1, _, _ = _fake_ensemble([zs[0], zs[0]], 0b11)         # two identical models == one
    assert np.allclose(p1, oracle.softmax(zs[0]), atol=1e-15)
    pa, _, _ = _fake_ensemble(zs, 0b111)                     # model order does not matter
    pb, _, _ = _fake_ensemble(zs[::-1], 0b111)
    assert np.allclose(pa, pb, atol=1e-15)
    assert np.allclose(pa.sum(1), 1.0, atol=1e-14)


def test_mask_validation_counts():
    """Exactly 2**|M| - 1 masks are valid (v = 0 excluded, Section 5.2)."""
    zs = [rng.standard_normal((2, 3)) for _ in range(3)]
    ok = 0
    for mask in range(0, 1 << 4):
        try:
            _fake_ensemble(zs, mask)
            ok += 1
        except ValueError:
            pass
    assert ok == 2 ** 3 - 1


# ---------------------------------------------------------------- bf16 rounding
def test_bf16_rounding_ties_to_even():
    vals = np.array([1.0, 1 + 2 ** -8, 1 + 3 * 2 ** -8, 1 + 2 ** -8 + 2 ** -20, -(1 + 2 ** -8),
                     3.0, 0.1, 2 ** -130 * 1.5 * 2 ** 10])
    want = np.array([1.0, 1.0, 1 + 2 ** -6, 1 + 2 ** -7, -1.0, 3.0, 0.10009765625, 2 ** -120 * 1.5])
    assert np.array_equal(oracle.to_bf16_rne(vals), want)
    # agrees with torch's float32 -> bfloat16 cast on float32-representable inputs
    x = rng.standard_normal(10000).astype(np.float32).astype(np.float64)
    tb = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(oracle.to_bf16_rne(x), tb)


def test_generator_rounding_agrees_with_torch():
    x = rng.standard_normal(10000).astype(np.float32) * 7
    tb = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(wl.round_bf16_rne_f32(x), tb)


# ---------------------------------------------------------------- architecture wiring
def test_published_parameter_counts():
    assert wl.resnet50().param_count() == 25_557_032
    assert wl.resnet101().param_count() == 44_549_160
    assert wl.vgg16().param_count() == 138_357_544
    assert wl.textcnn().param_count() == 9_360_902
    assert wl.toy_cnn().param_count(count_bn_affine=False) == 5_370
    assert wl.toy_cnn().param_count() - wl.toy_cnn().param_count(False) == 96


def test_mac_counts():
    assert abs(oracle.model_macs(wl.resnet50()) / 4.09e9 - 1) < 0.01
    assert abs(oracle.model_macs(wl.resnet101()) / 7.80e9 - 1) < 0.01
    assert abs(oracle.model_macs(wl.vgg16()) / 15.47e9 - 1) < 0.005
    assert oracle.model_macs(wl.toy_cnn()) == 32 * 32 * 16 * 27 + 16 * 16 * 32 * 144 + 320


def test_tiny_resnet_block_brute():
    """Conv+BN+ReLU -> conv+BN + residual -> ReLU through run_model vs scalar loops."""
    L = wl.Layer
    spec = wl.ModelSpec("blk", [
        L(op=wl.CONV2D, input=-1, c_in=2, c_out=2, kh=3, kw=3, stride=1, pad=1, relu=True, bn=True),
        L(op=wl.CONV2D, input=0, input2=-1, c_in=2, c_out=2, kh=3, kw=3, stride=1, pad=1, relu=True, bn=True),
    ], 2, (2, 4, 4))
    # residual of the model input: express it with an identity 1x1 conv first
    spec.layers.insert(0, L(op=wl.CONV2D, input=-1, c_in=2, c_out=2, kh=1, kw=1, relu=False))
    spec.layers[1].input = -1
    spec.layers[2].input = 1
    spec.layers[2].input2 = 0
    P = wl.gen_params(spec, 7, False, "random")
    P.layers[0].weight = np.eye(2, dtype=np.float32).reshape(2, 2, 1, 1)
    x = rng.standard_normal((1, 2, 4, 4))
    got = oracle.run_model(spec, P, x)
    def bn(v, lp, c):
        return (v - lp.bn_mean[c]) / math.sqrt(lp.bn_var[c] + lp.bn_eps) * lp.bn_gamma[c] + lp.bn_beta[c]
    a = brute.conv2d(x.tolist(), P.layers[1].weight.tolist(), 1, 1)
    a = [[[[max(0.0, bn(a[0][c][i][j], P.layers[1], c)) for j in range(4)] for i in range(4)] for c in range(2)]]
    b = brute.conv2d(a, P.layers[2].weight.tolist(), 1, 1)
    ref = [[[[max(0.0, bn(b[0][c][i][j], P.layers[2], c) + x[0, c, i, j]) for j in range(4)] for i in range(4)]
            for c in range(2)]]
    assert np.allclose(got, np.array(ref), atol=1e-12)


# ---------------------------------------------------------------- majority vote (Section 5.2)
def test_vote_golden_example():
    g = json.load(open(os.path.join(GOLDEN, "vote_3x4.json")))
    logits = [np.array(z) for z in g["logits"]]
    assert [oracle.argmax_first(z).tolist() for z in logits] == g["model_predictions"]
    v, lab = oracle.combine_vote(logits)
    assert np.allclose(v, g["expected_votes"], atol=1e-15)
    assert lab.tolist() == g["expected_labels"]


def test_vote_invariants():
    zs = [rng.standard_normal((50, 7)) for _ in range(4)]
    v, lab = oracle.combine_vote(zs[:1])                  # one model: its own argmax, one vote
    assert np.array_equal(lab, np.argmax(zs[0], 1)) and np.allclose(v.sum(1), 1.0)
    v, lab = oracle.combine_vote([zs[0], zs[0], zs[1]])   # a duplicated model is a majority
    assert np.array_equal(lab, np.argmax(zs[0], 1))
    v, lab = oracle.combine_vote(zs)
    assert np.allclose(v.sum(1), 1.0, atol=1e-15)
    # the winner always has the maximal vote count
    assert np.all(v[np.arange(50), lab] == v.max(1))
    # brute force over priorities: with two models that disagree, the first model wins
    a, b = np.zeros((1, 3)), np.zeros((1, 3))
    a[0, 2] = 1.0
    b[0, 0] = 1.0
    assert oracle.combine_vote([a, b])[1][0] == 2 and oracle.combine_vote([b, a])[1][0] == 0


def test_vote_two_models_equal_the_priority_model():
    """Section 5.2 observes that a two-model ensemble predicts exactly what its more
    accurate member predicts: with two voters every disagreement is a tie."""
    za, zb = rng.standard_normal((200, 10)), rng.standard_normal((200, 10))
    assert (np.argmax(za, 1) != np.argmax(zb, 1)).sum() > 100
    assert np.array_equal(oracle.combine_vote([za, zb])[1], np.argmax(za, 1))
    assert np.array_equal(oracle.combine_vote([zb, za])[1], np.argmax(zb, 1))


def test_tiny_textcnn_brute():
    """Embedding -> three conv1d max-over-time branches -> concatenations -> FC through
    run_model vs scalar loops: the table gather as list indexing, each branch through
    the scalar conv1d, the joins as explicit list concatenation in width order, then the
    scalar FC.  Non-zero biases and unequal widths make any mis-wiring visible."""
    spec = wl.textcnn(vocab=11, seq_len=9, dim=3, filters=2, widths=(2, 3, 4), n_classes=3)
    P = wl.gen_params(spec, 5, False, "random")
    r = np.random.default_rng(12)
    for lp in P.layers:
        if lp.bias is not None:
            lp.bias = r.standard_normal(lp.bias.shape).astype(np.float32)
    tok = r.integers(0, 11, size=(2, 9)).astype(np.int32)
    got = oracle.run_model(spec, P, tok)
    table = P.layers[0].weight.tolist()
    emb = [[table[t] for t in row] for row in tok.tolist()]
    branches = [brute.conv1d_maxtime(emb, P.layers[i].weight.tolist(), P.layers[i].bias.tolist(), True)
                for i in (1, 2, 3)]
    feats = [branches[0][n] + branches[1][n] + branches[2][n] for n in range(2)]
    ref = brute.fc(feats, P.layers[-1].weight.tolist(), P.layers[-1].bias.tolist())
    assert got.shape == (2, 3)
    assert np.allclose(got, np.array(ref), atol=1e-12)
    # a wrong join order is visible at this size
    swapped = [branches[1][n] + branches[0][n] + branches[2][n] for n in range(2)]
    assert not np.allclose(got, np.array(brute.fc(swapped, P.layers[-1].weight.tolist(),
                                                  P.layers[-1].bias.tolist())), atol=1e-6)


def test_concat_brute():
    a = rng.standard_normal((3, 4))
    b = rng.standard_normal((3, 2))
    ref = [list(a[i]) + list(b[i]) for i in range(3)]
    assert np.array_equal(oracle.concat(a, b), np.array(ref))

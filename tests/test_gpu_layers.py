"""Single-layer parity through the C ABI.

Each probe model is the layer(s) under test followed by an FC whose weight is the
identity, so the model's logits are the stored output tensor flattened in (c, h, w)
order (with bf16 storage the identity FC is exact: one nonzero product per output,
accumulated in fp32).  Shapes cover the edge cases of the kernels: input channels
not a multiple of 8 or 64, odd and non-square images, stride 2, 1x1 and 7x7 kernels,
channel counts that leave a ragged tile, residual adds, split-K FCs and a small
TextCNN.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from workloads import Layer, ModelSpec, CONV2D, MAXPOOL2D, GLOBAL_AVGPOOL, FC, EMBEDDING, CONV1D_MAXTIME, CONCAT
from paper_1804_06087_amd import Ensemble

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def probe(layers, in_shape, out_elems, identity=True, n_out=None, seed=5, bf16=True, vocab=0):
    L = list(layers)
    n_out = out_elems if identity else n_out
    L.append(Layer(op=FC, input=len(layers) - 1, c_in=out_elems, c_out=n_out, bias=True))
    spec = ModelSpec("probe", L, n_out, in_shape, vocab=vocab)
    params = wl.gen_params(spec, seed, bf16, "random")
    if identity:
        params.layers[-1].weight = np.eye(out_elems, dtype=np.float32)
    return spec, params


def gpu_logits(spec, params, batch, precision):
    n = batch.shape[0]
    with Ensemble([spec], [params], precision=precision, max_batch=n) as ens:
        x = torch.from_numpy(batch).to(DEV)
        out = torch.empty((n, spec.n_classes), dtype=torch.float32, device=DEV)
        ens.model_logits(0, x, n, out)
        torch.cuda.synchronize()
        return out.cpu().numpy()


def check_bf16_tensor(z, ref):
    """bf16-stored tensors: each element within one bf16 step of the oracle's
    (fp32 vs fp64 accumulation may round the other way), few elements differing."""
    ref = np.asarray(ref, np.float64)
    d = np.abs(z - ref)
    tol = np.abs(ref) * 2.0 ** -7 + 1e-6 * np.abs(ref).max()
    assert (d <= tol).all(), f"max excess {(d - tol).max()}"
    assert (d > 0).mean() < 0.02, f"{(d > 0).mean():.3%} of elements differ"


def conv(i, c_in, c_out, k, s=1, p=None, relu=True, bn=True, bias=False, res=-1):
    return Layer(op=CONV2D, input=i, input2=res, c_in=c_in, c_out=c_out, kh=k, kw=k, stride=s,
                 pad=k // 2 if p is None else p, relu=relu, bn=bn, bias=bias)


CASES = {
    # name: (layers, input (C, H, W), n, output elements)
    "stem3x3_cin3": ([conv(-1, 3, 16, 3)], (3, 7, 7), 3, 16 * 7 * 7),
    "s2_cin24_cout40_nonsquare": ([conv(-1, 24, 40, 3, s=2)], (24, 11, 7), 5, 40 * 6 * 4),
    "1x1_s2_cout136": ([conv(-1, 64, 136, 1, s=2, p=0)], (64, 4, 4), 4, 136 * 2 * 2),
    "7x7_s2_p3_stem": ([conv(-1, 3, 64, 7, s=2, p=3)], (3, 7, 7), 2, 64 * 4 * 4),
    "residual_block": ([conv(-1, 16, 32, 1, p=0, relu=False), conv(-1, 16, 32, 3, res=0)], (16, 5, 5), 3,
                       32 * 5 * 5),
    "vgg_style_bias_no_bn": ([conv(-1, 8, 32, 3, bn=False, bias=True)], (8, 6, 5), 3, 32 * 6 * 5),
    "maxpool3_s2_p1_odd": ([conv(-1, 8, 16, 3), Layer(op=MAXPOOL2D, input=0, c_in=16, c_out=16, kh=3, kw=3,
                                                       stride=2, pad=1)], (8, 9, 9), 2, 16 * 5 * 5),
    "maxpool2_s2": ([conv(-1, 8, 16, 3), Layer(op=MAXPOOL2D, input=0, c_in=16, c_out=16, kh=2, kw=2, stride=2)],
                    (8, 8, 6), 2, 16 * 4 * 3),
    "gap": ([conv(-1, 8, 48, 3), Layer(op=GLOBAL_AVGPOOL, input=0, c_in=48, c_out=48)], (8, 7, 5), 6, 48),
    "many_tiles_ragged_m": ([conv(-1, 32, 16, 3)], (32, 7, 9), 37, 16 * 7 * 9),
    # several 64-channel blocks under a 3x3 kernel: the bf16 kernel's channel-block K
    # order, the fp32 kernel's (tap, channel) order
    "cin192_3x3": ([conv(-1, 192, 24, 3)], (192, 5, 6), 3, 24 * 5 * 6),
    # image-input convolutions with few channels (input padded to 8 storage channels)
    "stem_3x3_cout32_ragged": ([conv(-1, 3, 32, 3)], (3, 5, 6), 7, 32 * 5 * 6),
    "stem_7x7_s2_cout128": ([conv(-1, 3, 128, 7, s=2, p=3)], (3, 4, 4), 3, 128 * 2 * 2),
    "stem_1ch_5x5_cout96": ([conv(-1, 1, 96, 5, p=2, bn=False, bias=True)], (1, 3, 3), 5, 96 * 3 * 3),
    # 2x2 stride-2 max-pool fused into the conv epilogue (bf16): ragged window count,
    # 64 storage channels; a long-K conv whose tiny output is split over K (the pooled
    # split-K reduction); an odd-sized conv output that is pooled separately (floor)
    "pool2_fused_ragged": ([conv(-1, 64, 24, 3), Layer(op=MAXPOOL2D, input=0, c_in=24, c_out=24, kh=2, kw=2,
                                                        stride=2)], (64, 10, 14), 3, 24 * 5 * 7),
    "pool2_fused_split_k": ([conv(-1, 512, 64, 3), Layer(op=MAXPOOL2D, input=0, c_in=64, c_out=64, kh=2, kw=2,
                                                          stride=2)], (512, 4, 4), 2, 64 * 2 * 2),
    "pool2_odd_unfused": ([conv(-1, 8, 16, 3), Layer(op=MAXPOOL2D, input=0, c_in=16, c_out=16, kh=2, kw=2,
                                                      stride=2)], (8, 7, 9), 3, 16 * 3 * 4),
    # output maps of a multiple of 128 pixels, pooled to keep the probe small
    "stem_window_3x3": ([conv(-1, 3, 32, 3), Layer(op=MAXPOOL2D, input=0, c_in=32, c_out=32, kh=4, kw=4, stride=4)],
                        (3, 16, 16), 3, 32 * 4 * 4),
    "stem_window_7x7_s2": ([conv(-1, 3, 64, 7, s=2, p=3),
                            Layer(op=MAXPOOL2D, input=0, c_in=64, c_out=64, kh=4, kw=4, stride=4)],
                           (3, 32, 32), 2, 64 * 4 * 4),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_layer_bf16(name):
    layers, shape, n, out_elems = CASES[name]
    spec, params = probe(layers, shape, out_elems)
    batch = wl.gen_images(n, shape, "normal", True, seed=11)
    z = gpu_logits(spec, params, batch, "bf16")
    ref = oracle.run_model(spec, params, batch, act="bf16")
    check_bf16_tensor(z, ref)


@pytest.mark.parametrize("name", ["stem3x3_cin3", "s2_cin24_cout40_nonsquare", "residual_block", "maxpool3_s2_p1_odd",
                                  "gap", "7x7_s2_p3_stem", "cin192_3x3", "pool2_fused_split_k", "maxpool2_s2",
                                  "pool2_fused_ragged", "pool2_odd_unfused"])
def test_layer_fp32(name):
    layers, shape, n, out_elems = CASES[name]
    spec, params = probe(layers, shape, out_elems, bf16=False)
    batch = wl.gen_images(n, shape, "normal", False, seed=11)
    z = gpu_logits(spec, params, batch, "fp32")
    ref = oracle.run_model(spec, params, batch)
    assert np.abs(z - ref).max() <= 1e-5 * np.abs(ref).max()


@pytest.mark.parametrize("precision", ["bf16", "fp32"])
def test_fc_flatten_order_and_split_k(precision):
    """FC on a spatial input (flattened in (c, h, w) order) with a long K that the bf16
    path splits across workgroups; random weights, fp32 logits."""
    bf = precision == "bf16"
    layers = [conv(-1, 16, 64, 1, p=0)]                    # -> [64, 8, 8] = 4096 features
    spec, params = probe(layers, (16, 8, 8), 64 * 8 * 8, identity=False, n_out=100)
    params = wl.gen_params(spec, 9, bf, "random")
    for n in (1, 3, 70):
        batch = wl.gen_images(n, (16, 8, 8), "normal", bf, seed=3)
        z = gpu_logits(spec, params, batch, precision)
        ref = oracle.run_model(spec, params, batch, act="bf16" if bf else None)
        err = np.abs(z - ref).max() / np.abs(ref).max()
        assert err <= (1e-4 if bf else 1e-5), (n, err)


def test_textcnn_small():
    spec = wl.textcnn(vocab=50, seq_len=12, dim=20, filters=5, widths=(2, 3, 5), n_classes=2)
    for precision in ("bf16", "fp32"):
        bf = precision == "bf16"
        params = wl.gen_params(spec, 4, bf, "random")
        for L, P in zip(spec.layers, params.layers):       # non-zero biases exercise the epilogue
            if L.bias:
                P.bias = np.linspace(-0.2, 0.3, L.c_out).astype(np.float32)
        tok = wl.gen_tokens(9, 12, 50, seed=2)
        z = gpu_logits(spec, params, tok, precision)
        ref = oracle.run_model(spec, params, tok, act="bf16" if bf else None)
        err = np.abs(z - ref).max() / np.abs(ref).max()
        assert err <= (1e-2 if bf else 1e-5), (precision, err)


def test_textcnn_long_sequence():
    """Long sequences (260 tokens; 258 and 254 positions for widths 3 and 7, so a
    position range spans several row tiles and the max over time many of them), odd
    channel counts and a batch that is not a multiple of anything."""
    spec = wl.textcnn(vocab=64, seq_len=260, dim=24, filters=12, widths=(3, 7), n_classes=2)
    params = wl.gen_params(spec, 6, True, "random")
    for L, P in zip(spec.layers, params.layers):
        if L.bias:
            P.bias = np.linspace(-0.3, 0.2, L.c_out).astype(np.float32)
    tok = wl.gen_tokens(5, 260, 64, seed=8)
    z = gpu_logits(spec, params, tok, "bf16")
    ref = oracle.run_model(spec, params, tok, act="bf16")
    err = np.abs(z - ref).max() / np.abs(ref).max()
    assert err <= 1e-2, err


def _branch_probe(dim, seq_len, filters, widths, vocab=97, extra_reader=False, seed=11, relu=True):
    """Embedding, conv1d max-over-time branches of the given widths and filter
    counts, their concatenation in order, then the identity FC: the logits are the
    concatenated feature vector.  With extra_reader, the first branch is also
    concatenated a second time, so that it has two readers and must not be fused."""
    L = [Layer(op=EMBEDDING, input=-1, c_in=vocab, c_out=dim)]
    feats = []
    for f, w in zip(filters, widths):
        L.append(Layer(op=CONV1D_MAXTIME, input=0, c_in=dim, c_out=f, kh=1, kw=w, relu=relu, bias=True))
        feats.append(len(L) - 1)
    x, c = feats[0], filters[0]
    for fi, f in zip(feats[1:], filters[1:]):
        L.append(Layer(op=CONCAT, input=x, input2=fi, c_in=c, c_out=c + f))
        x, c = len(L) - 1, c + f
    if extra_reader:
        L.append(Layer(op=CONCAT, input=x, input2=feats[0], c_in=c, c_out=c + filters[0]))
        c += filters[0]
    spec, params = probe(L, (seq_len,), c, seed=seed, vocab=vocab)
    for Lr, P in zip(spec.layers, params.layers):
        if Lr.bias and Lr.op == CONV1D_MAXTIME:
            P.bias = np.linspace(-0.3, 0.2, Lr.c_out).astype(np.float32)
    return spec, params


def _run_traced(spec, params, tok, cfg=-1):
    """Logits and traced kernel kinds of one forward pass (cfg >= 0: forced tile)."""
    n = tok.shape[0]
    with Ensemble([spec], [params], precision="bf16", max_batch=n) as ens:
        if cfg >= 0:
            ens.force_tile(cfg)
        x = torch.from_numpy(tok).to(DEV)
        out = torch.empty((n, spec.n_classes), dtype=torch.float32, device=DEV)
        ens.model_logits(0, x, n, out)          # tunes the tiles; a second call must agree
        torch.cuda.synchronize()
        first = out.cpu().numpy()
        ens.trace(True)
        ens.model_logits(0, x, n, out)
        torch.cuda.synchronize()
        z = out.cpu().numpy()
        assert np.array_equal(z.view(np.uint32), first.view(np.uint32)), "repeated call differs"
        return z, [r["kind"] for r in ens.trace_read()]


# Batches large enough that neither the fused GEMM nor any separate branch splits K
# (a split sums a row's products in parts, which the two layouts cut differently).
@pytest.mark.parametrize("n, case", [
    (72, dict(dim=300, seq_len=256, filters=(100, 100, 100), widths=(3, 4, 5))),  # TextCNN: aligned K, 64-row blocks
    (384, dict(dim=128, seq_len=50, filters=(70, 90), widths=(2, 6))),           # aligned, tiles mixing widths
    (570, dict(dim=64, seq_len=33, filters=(13, 21, 6), widths=(5, 2, 3))),      # aligned, one 64-row block
    (130, dict(dim=64, seq_len=130, filters=(64, 64), widths=(2, 3))),           # max in the epilogue, 129 positions
    (72, dict(dim=300, seq_len=256, filters=(100, 100, 100), widths=(3, 4, 5), relu=False)),  # negative maxima
    (460, dict(dim=70, seq_len=40, filters=(13, 21, 6), widths=(5, 2, 3))),      # unaligned K, ragged segments
    (7, dict(dim=24, seq_len=30, filters=(5, 7, 9), widths=(2, 3, 4), extra_reader=True)),   # not fusable
])
def test_fused_branches_bitwise(n, case, monkeypatch):
    """Sibling max-over-time convolutions joined by concatenation run as one GEMM and
    one segmented max: the feature vector is bitwise that of the separate branches
    (RAFIKI_FUSE_BRANCHES=0) and within one bf16 step of the oracle's."""
    spec, params = _branch_probe(**case)
    tok = wl.gen_tokens(n, case["seq_len"], 97, seed=3)
    fused, kf = _run_traced(spec, params, tok)
    monkeypatch.setenv("RAFIKI_FUSE_BRANCHES", "0")
    separate, ks = _run_traced(spec, params, tok)
    nb = len(case["widths"])
    assert ks.count("concat") == nb - 1 + (1 if case.get("extra_reader") else 0)
    assert ks.count("pool") == nb
    assert "splitk_reduce" not in ks and "splitk_reduce" not in kf
    if case.get("extra_reader"):
        assert kf == ks
    else:
        assert kf.count("concat") == 0 and kf.count("pool") == 1
        assert kf.count("conv_mfma") == ks.count("conv_mfma") - (nb - 1)
        # with 64-aligned storage channels the GEMM gathers the embedding rows itself
        assert kf.count("embed") == (0 if case["dim"] % 64 == 0 or case["dim"] == 300 else 1)
    assert ks.count("embed") == 1
    assert np.array_equal(fused.view(np.uint32), separate.view(np.uint32))
    ref = oracle.run_model(spec, params, tok, act="bf16")
    check_bf16_tensor(fused, ref)


@pytest.mark.parametrize("n, case", [
    (7, dict(dim=300, seq_len=256, filters=(100, 100, 100), widths=(3, 4, 5))),
    (1, dict(dim=300, seq_len=256, filters=(100, 100, 100), widths=(3, 4, 5))),
    (72, dict(dim=300, seq_len=256, filters=(100, 100, 100), widths=(3, 4, 5))),    # unsplit: max in the epilogue
    (72, dict(dim=300, seq_len=256, filters=(100, 100, 100), widths=(3, 4, 5), relu=False)),
    (130, dict(dim=64, seq_len=130, filters=(64, 64), widths=(2, 3))),
    (9, dict(dim=128, seq_len=50, filters=(70, 90), widths=(2, 6))),
    (7, dict(dim=24, seq_len=9, filters=(8, 16), widths=(9, 1))),              # a branch as wide as the sequence
])
def test_fused_branches_tile_independent(n, case):
    """Whichever tile runs the fused GEMM (each skips the taps its rows lack; at small
    batches it splits K, at large ones with long sequences it takes the max in its
    epilogue), the feature vector is the same bit for bit, and within one bf16 step
    of the oracle's; repeated calls on one handle agree too (the epilogue's slots are
    reset as they are read)."""
    spec, params = _branch_probe(**case)
    tok = wl.gen_tokens(n, case["seq_len"], 97, seed=4)
    base, kinds = _run_traced(spec, params, tok)
    assert kinds.count("concat") == 0 and kinds.count("pool") == 1
    assert kinds.count("embed") == (0 if case["dim"] % 64 == 0 or case["dim"] == 300 else 1)
    for cfg in (8, 6, 5, 3, 16, 38, 40):      # 64x64, 64x128, 128x128, 128x256, 128x256, 256x64, 128x128
        z, _ = _run_traced(spec, params, tok, cfg)
        assert np.array_equal(z.view(np.uint32), base.view(np.uint32)), cfg
    ref = oracle.run_model(spec, params, tok, act="bf16")
    check_bf16_tensor(base, ref)


def test_invalid_token_ids_read_zero_rows(monkeypatch):
    """Token ids outside [0, vocab) read a zero embedding row, both in the embedding
    kernel (branches apart) and in the GEMM that gathers the rows itself (fused)."""
    import copy
    case = dict(dim=128, seq_len=50, filters=(70, 90), widths=(2, 6))
    spec, params = _branch_probe(**case)
    vocab = spec.layers[0].c_in
    tok = wl.gen_tokens(384, case["seq_len"], vocab, seed=5)
    rng = np.random.default_rng(9)
    bad = rng.random(tok.shape) < 0.05
    tok[bad] = rng.choice(np.array([-1, vocab, vocab + 7, 2**31 - 1, -2**31], dtype=np.int64),
                          size=int(bad.sum())).astype(np.int32)
    fused, kf = _run_traced(spec, params, tok)
    assert kf.count("embed") == 0
    monkeypatch.setenv("RAFIKI_FUSE_BRANCHES", "0")
    separate, ks = _run_traced(spec, params, tok)
    assert ks.count("embed") == 1
    assert np.array_equal(fused.view(np.uint32), separate.view(np.uint32))
    p2 = copy.deepcopy(params)
    p2.layers[0].weight = np.vstack([params.layers[0].weight, np.zeros((1, case["dim"]), np.float32)])
    ref = oracle.run_model(spec, p2, np.where(bad, vocab, tok), act="bf16")
    check_bf16_tensor(fused, ref)

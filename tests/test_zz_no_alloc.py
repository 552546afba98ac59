"""rafiki_ensemble_infer_noalloc against rafiki_ensemble_infer, through the C ABI.

The no-alloc variant runs the same kernels in the same order with its split-K
partial sums and epilogue-max keys in the library's static device array, so its
outputs must be bitwise those of infer; they are also checked against the fp64
oracle.  Each case makes two calls in a row, the second with a smaller batch, so
that the second call meets what the first left in the shared array.
"""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from workloads import Layer, ModelSpec, FC
from paper_1804_06087_amd import Ensemble, RafikiError, RAFIKI_ERR_UNSUPPORTED

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def _both(ens, x, n, mask, C):
    out = []
    for fn in (ens.infer, ens.infer_noalloc):
        probs = torch.full((n, C), -1.0, dtype=torch.float32, device=DEV)
        labels = torch.full((n,), -7, dtype=torch.int32, device=DEV)
        fn(x, n, mask, probs, labels)
        torch.cuda.synchronize()
        out.append((probs.cpu().numpy(), labels.cpu().numpy()))
    return out


def _oracle_check(specs, params, batch, n, mask, p, lab):
    p_ref, _, _ = oracle.ensemble(specs, params, batch[:n], mask, act="bf16")
    srt = np.sort(p_ref, 1)
    excused = (srt[:, -1] - srt[:, -2]) < 1e-3
    assert not ((lab != oracle.argmax_first(p_ref)) & ~excused).any()
    assert np.allclose(p.sum(1), 1.0, atol=1e-5)


def test_noalloc_resnet50_split_k_two_calls():
    """ResNet-50 at n = 8 and then 3: its 7x7 layers and FC split K (partials in the
    static array)."""
    cfg, specs, params, batch = wl.build_config(4, n=8, models=[0])
    with Ensemble(specs, params, precision="bf16", max_batch=8) as ens:
        x = torch.from_numpy(batch).to(DEV)
        for n in (8, 3):
            (p0, l0), (p1, l1) = _both(ens, x, n, 0b1, 1000)
            assert np.array_equal(p0, p1) and np.array_equal(l0, l1), n
            _oracle_check(specs, params, batch, n, 0b1, p1, l1)


def test_noalloc_textcnn_epilogue_max_two_calls():
    """Two TextCNNs at n = 32 and then 24 (the fused branches take the max over time
    in the GEMM epilogue, keys in the static array), then n = 5 (split K)."""
    cfg, specs, params, batch = wl.build_config(5, n=32, models=[0, 1])
    with Ensemble(specs, params, precision="bf16", max_batch=32) as ens:
        x = torch.from_numpy(batch).to(DEV)
        for n in (32, 24, 5):
            (p0, l0), (p1, l1) = _both(ens, x, n, 0b11, 2)
            assert np.array_equal(p0, p1) and np.array_equal(l0, l1), n
            _oracle_check(specs, params, batch, n, 0b11, p1, l1)
            # which path ran: unsplit fused GEMMs (maxima in the epilogue) at n >= 24
            ens.trace(True)
            probs = torch.empty((n, 2), dtype=torch.float32, device=DEV)
            labels = torch.empty((n,), dtype=torch.int32, device=DEV)
            ens.infer_noalloc(x, n, 0b11, probs, labels)
            torch.cuda.synchronize()
            recs = ens.trace_read()
            ens.trace(False)
            split = [r["splits"] for r in recs if r["kind"] == "conv_mfma" and r["flops"] > 1e9 * n / 64]
            assert split and all(s == (1 if n >= 24 else split[0]) for s in split), (n, split)
            assert (n >= 24) == all(s == 1 for s in split), (n, split)
            assert np.array_equal(probs.cpu().numpy(), p1) and np.array_equal(labels.cpu().numpy(), l1)


def test_noalloc_rejects_oversize_scratch():
    """Five FC models whose split-K partials need 16 MiB each at n = 256: 80 MiB is
    beyond the 64 MiB array, so the call fails before enqueueing anything; a call
    that fits still matches infer afterwards."""
    c_in, C = 16384, 1024
    spec = ModelSpec("wide_fc", [Layer(op=FC, input=-1, c_in=c_in, c_out=C, bias=True)], C, (c_in, 1, 1))
    specs = [spec] * 5
    params = [wl.gen_params(spec, 11 + i, True, "random") for i in range(5)]
    batch = wl.gen_images(256, (c_in, 1, 1), "normal", True)
    with Ensemble(specs, params, precision="bf16", max_batch=256) as ens:
        x = torch.from_numpy(batch).to(DEV)
        probs = torch.empty((256, C), dtype=torch.float32, device=DEV)
        labels = torch.empty((256,), dtype=torch.int32, device=DEV)
        with pytest.raises(RafikiError) as ei:
            ens.infer_noalloc(x, 256, 0b11111, probs, labels)
        assert ei.value.code == RAFIKI_ERR_UNSUPPORTED
        (p0, l0), (p1, l1) = _both(ens, x, 64, 0b00111, C)
        assert np.array_equal(p0, p1) and np.array_equal(l0, l1)

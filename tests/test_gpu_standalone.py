"""The path's memory-bound kernels called on their own through the C ABI
(rafiki_combine_mean / _vote, rafiki_maxpool_nhwc_bf16, rafiki_global_avgpool_nhwc_bf16)
against the oracle: ragged row counts, odd class counts, the 32-model limit, pooling
with and without padding, and the argument checks."""
import numpy as np
import pytest
import torch

import oracle
import workloads as wl
from paper_1804_06087_amd import RafikiError, RAFIKI_ERR_INVALID
from paper_1804_06087_amd.binding import combine_mean, combine_vote, maxpool_nhwc_bf16, global_avgpool_nhwc_bf16

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


def labels_vs_oracle(lab, p_ref):
    """Labels equal the oracle's first-index argmax of its fp64 mean probabilities,
    except where its top-2 differ by < 1e-3; there the label must be within 1e-3 of
    the top."""
    srt = np.sort(p_ref, 1)
    ref = oracle.argmax_first(p_ref)
    mism = np.nonzero(lab != ref)[0]
    assert ((srt[mism, -1] - srt[mism, -2]) < 1e-3).all(), f"label mismatches at rows {mism}"
    assert (p_ref[mism, lab[mism]] >= srt[mism, -1] - 1e-3).all()


@pytest.mark.parametrize("S,n,C", [(3, 37, 1000), (1, 5, 10), (32, 9, 7), (2, 130, 1024)])
def test_combine_mean_and_vote(S, n, C):
    rng = np.random.Generator(np.random.PCG64(S * 1000 + n))
    z = (rng.standard_normal((S, n, C)) * 3).astype(np.float32)
    z[:, 0, :] = 0.5                                  # a row of exact ties
    zt = torch.from_numpy(z).to(DEV)
    p = torch.empty((n, C), dtype=torch.float32, device=DEV)
    lab = torch.empty((n,), dtype=torch.int32, device=DEV)
    combine_mean(zt, p, lab)
    torch.cuda.synchronize()
    p_ref = oracle.combine_mean([oracle.softmax(z[s].astype(np.float64)) for s in range(S)])
    assert np.abs(p.cpu().numpy() - p_ref).max() <= 1e-6
    labels_vs_oracle(lab.cpu().numpy(), p_ref)
    assert lab[0].item() == 0                         # exact ties: the lowest index
    v = torch.empty((n, C), dtype=torch.float32, device=DEV)
    combine_vote(zt, v, lab)
    torch.cuda.synchronize()
    v_ref, l_ref = oracle.combine_vote([z[s] for s in range(S)])
    assert np.abs(v.cpu().numpy() - v_ref).max() <= 1e-6     # count * fp32(1/S)
    assert np.array_equal(lab.cpu().numpy(), l_ref)


def test_combine_unaligned_buffers():
    """Buffers that start 4 bytes past a 16-byte boundary take the scalar path."""
    S, n, C = 3, 21, 1000
    rng = np.random.Generator(np.random.PCG64(77))
    z = (rng.standard_normal((S, n, C)) * 3).astype(np.float32)
    zbuf = torch.empty(S * n * C + 1, dtype=torch.float32, device=DEV)
    zt = zbuf[1:].view(S, n, C)
    zt.copy_(torch.from_numpy(z))
    pbuf = torch.empty(n * C + 1, dtype=torch.float32, device=DEV)
    p = pbuf[1:].view(n, C)
    lab = torch.empty((n,), dtype=torch.int32, device=DEV)
    combine_mean(zt, p, lab)
    torch.cuda.synchronize()
    p_ref = oracle.combine_mean([oracle.softmax(z[s].astype(np.float64)) for s in range(S)])
    assert np.abs(p.cpu().numpy() - p_ref).max() <= 1e-6
    labels_vs_oracle(lab.cpu().numpy(), p_ref)
    combine_vote(zt, p, lab)
    torch.cuda.synchronize()
    v_ref, l_ref = oracle.combine_vote([z[s] for s in range(S)])
    assert np.abs(p.cpu().numpy() - v_ref).max() <= 1e-6
    assert np.array_equal(lab.cpu().numpy(), l_ref)


def _nhwc_bf16(n, h, w, c, seed):
    x = wl.round_bf16_rne_f32(np.random.Generator(np.random.PCG64(seed)).standard_normal((n, h, w, c))
                              .astype(np.float32))
    return x, torch.from_numpy(x).to(DEV).to(torch.bfloat16)


@pytest.mark.parametrize("shape,k,s,p", [((3, 9, 11, 16), 3, 2, 1), ((2, 8, 6, 64), 2, 2, 0),
                                         ((1, 5, 5, 8), 5, 1, 2), ((4, 13, 7, 24), 3, 3, 0),
                                         ((2, 10, 10, 8), 3, 2, 0), ((1, 112, 112, 64), 3, 2, 1),
                                         ((2, 7, 13, 72), 3, 2, 1), ((3, 8, 5, 16), 3, 2, 2)])
def test_maxpool(shape, k, s, p):
    n, h, w, c = shape
    x, xt = _nhwc_bf16(n, h, w, c, seed=k * 10 + s)
    ho, wo = (h + 2 * p - k) // s + 1, (w + 2 * p - k) // s + 1
    y = torch.empty((n, ho, wo, c), dtype=torch.bfloat16, device=DEV)
    maxpool_nhwc_bf16(xt, y, k, s, p)
    torch.cuda.synchronize()
    ref = oracle.maxpool2d(x.transpose(0, 3, 1, 2).astype(np.float64), k, s, p).transpose(0, 2, 3, 1)
    assert np.array_equal(y.float().cpu().numpy(), ref.astype(np.float32))   # max is exact


@pytest.mark.parametrize("shape", [(3, 7, 7, 2048), (5, 1, 1, 8), (2, 16, 16, 24), (1, 254, 1, 104),
                                   (64, 7, 7, 2048), (70, 3, 5, 2048), (2048, 1, 3, 64)])
def test_global_avgpool(shape):
    n, h, w, c = shape
    x, xt = _nhwc_bf16(n, h, w, c, seed=h * w)
    y = torch.empty((n, c), dtype=torch.bfloat16, device=DEV)
    global_avgpool_nhwc_bf16(xt, y)
    torch.cuda.synchronize()
    ref = oracle.global_avgpool(x.transpose(0, 3, 1, 2).astype(np.float64))
    got = y.float().cpu().numpy()
    # fp32 sums, one bf16 rounding: within one bf16 step of the exact mean
    assert np.all(np.abs(got - ref) <= np.abs(ref) * 2.0 ** -8 + 1e-6), np.abs(got - ref).max()


def test_standalone_argument_errors():
    z = torch.zeros((33, 2, 4), dtype=torch.float32, device=DEV)
    p = torch.empty((2, 4), dtype=torch.float32, device=DEV)
    lab = torch.empty((2,), dtype=torch.int32, device=DEV)
    with pytest.raises(RafikiError) as e:
        combine_mean(z, p, lab)                          # more than 32 models
    assert e.value.code == RAFIKI_ERR_INVALID
    x = torch.zeros((1, 4, 4, 12), dtype=torch.bfloat16, device=DEV)
    y = torch.zeros((1, 2, 2, 12), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(RafikiError):
        maxpool_nhwc_bf16(x, y, 2, 2, 0)                 # channels not a multiple of 8
    x = torch.zeros((1, 4, 4, 8), dtype=torch.bfloat16, device=DEV)
    y = torch.zeros((1, 4, 4, 8), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(RafikiError):
        maxpool_nhwc_bf16(x, y, 2, 2, 2)                 # pad >= k
    with pytest.raises(ValueError):
        maxpool_nhwc_bf16(x, y, 2, 2, 0)                 # output buffer of the wrong shape
    with pytest.raises(ValueError):
        combine_mean(z[:3], p.to(torch.float64), lab)    # output of the wrong dtype


def test_mainloop_probe_checksums_and_arguments():
    """The main-loop probe (a diagnostic, not part of the path): its per-K-tile LDS writes
    go to chunks that no fragment read touches, so each wave's checksum is the same with
    and without them; every wave of every workgroup writes a finite checksum."""
    from paper_1804_06087_amd.binding import MAINLOOP_VARIANTS, probe_mainloop
    blocks = 300
    for v, (waves, *_rest) in MAINLOOP_VARIANTS.items():
        res = []
        for sync in (False, True):
            out = torch.full((blocks * 8,), float("nan"), dtype=torch.float32, device=DEV)
            probe_mainloop(v, sync, blocks, 5, out)
            torch.cuda.synchronize()
            o = out.view(blocks, 8)[:, :waves].cpu()
            assert torch.isfinite(o).all(), (v, sync)
            res.append(o)
        assert torch.equal(res[0], res[1]), v
    out = torch.empty((8,), dtype=torch.float32, device=DEV)
    for bad in ((4, False, 1, 1), (0, False, 0, 1), (0, True, 1, 0)):
        with pytest.raises(RafikiError) as e:
            probe_mainloop(*bad, out)
        assert e.value.code == RAFIKI_ERR_INVALID

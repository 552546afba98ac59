"""C-ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects invalid arguments with the documented status codes
(validation happens before any device call; without a device a valid create
returns RAFIKI_ERR_HIP instead of crashing)."""
import ctypes as C
import glob
import os
import re

import numpy as np
import pytest

import workloads as wl
import paper_1804_06087_amd as pkg
from paper_1804_06087_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        txt = open(h).read()
        names |= set(re.findall(r"^\s*(?:int|const char\*)\s+(rafiki_\w+)\s*\(", txt, re.M))
    return names


def test_header_declares_the_boundary():
    d = _declared()
    assert {"rafiki_ensemble_create", "rafiki_ensemble_infer", "rafiki_ensemble_destroy", "rafiki_last_error"} <= d


def test_library_exports_every_declared_symbol():
    lib = pkg.load_library()
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(pkg.EXPORTED) == _declared()


def _create(specs, params, precision=bd.RAFIKI_FP32, max_batch=8, n_models=None, opts_over=None, mutate=None):
    keep = []
    descs = (bd.RafikiModelDesc * len(specs))()
    arrs = []
    for i, (s, p) in enumerate(zip(specs, params)):
        arr = bd.make_layers(s, p, keep)
        arrs.append(arr)
        descs[i].n_layers = len(s.layers)
        descs[i].layers = C.cast(arr, C.POINTER(bd.RafikiLayer))
        descs[i].n_classes = s.n_classes
    if mutate:
        mutate(descs, arrs)
    o = bd.RafikiOpts()
    o.input_kind, o.c, o.h, o.w, o.vocab = 0, 3, 32, 32, 0
    o.precision, o.max_batch = precision, max_batch
    if opts_over:
        for k, v in opts_over.items():
            setattr(o, k, v)
    h = C.c_void_p(1234)
    rc = pkg.load_library().rafiki_ensemble_create(descs, len(specs) if n_models is None else n_models,
                                                   C.byref(o), C.byref(h))
    return rc, h


@pytest.fixture(scope="module")
def toy():
    cfg, specs, params, batch = wl.build_config(1)
    return specs, params


def test_null_arguments():
    lib = pkg.load_library()
    assert lib.rafiki_ensemble_create(None, 1, None, None) == bd.RAFIKI_ERR_INVALID
    assert "null" in bd.last_error()
    assert lib.rafiki_ensemble_destroy(None) == bd.RAFIKI_OK
    assert lib.rafiki_ensemble_infer(None, None, 1, 1, None, None, None) == bd.RAFIKI_ERR_INVALID
    assert lib.rafiki_ensemble_infer_vote(None, None, 1, 1, None, None, None) == bd.RAFIKI_ERR_INVALID
    assert lib.rafiki_ensemble_model_logits(None, 0, None, 1, None, None) == bd.RAFIKI_ERR_INVALID
    assert lib.rafiki_ensemble_info(None, None, None, None) == bd.RAFIKI_ERR_INVALID


@pytest.mark.parametrize("n_models", [0, 33])
def test_model_count_range(toy, n_models):
    rc, h = _create(*toy, n_models=n_models)
    assert rc == bd.RAFIKI_ERR_INVALID and h.value is None


@pytest.mark.parametrize("over", [{"precision": 7}, {"max_batch": 0}, {"input_kind": 9}, {"h": 0}])
def test_bad_options(toy, over):
    rc, h = _create(*toy, opts_over=over)
    assert rc == bd.RAFIKI_ERR_INVALID


def test_class_count_mismatch(toy):
    def m(descs, arrs):
        descs[1].n_classes = 9
    rc, _ = _create(*toy, mutate=m)
    assert rc == bd.RAFIKI_ERR_INVALID and "classes" in bd.last_error()


@pytest.mark.parametrize("field,value,needle", [
    ("input", 3, "input id"),          # forward reference
    ("c_in", 5, "channel"),            # conv channel mismatch
    ("stride", 0, "geometry"),
])
def test_malformed_layer(toy, field, value, needle):
    def m(descs, arrs):
        setattr(arrs[0][2], field, value)   # layer 2 = second conv of the toy CNN
    rc, _ = _create(*toy, mutate=m)
    assert rc == bd.RAFIKI_ERR_INVALID and needle in bd.last_error()


def test_last_layer_must_be_fc(toy):
    def m(descs, arrs):
        descs[0].n_layers = 4                # drop the FC
    rc, _ = _create(*toy, mutate=m)
    assert rc == bd.RAFIKI_ERR_INVALID and "last layer" in bd.last_error()


def test_partial_batchnorm_rejected(toy):
    def m(descs, arrs):
        arrs[0][0].bn_var = None
    rc, _ = _create(*toy, mutate=m)
    assert rc == bd.RAFIKI_ERR_INVALID and "batch-norm" in bd.last_error()


def test_valid_model_without_device_reports_hip_error(toy):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    rc, h = _create(*toy)
    assert rc == bd.RAFIKI_ERR_HIP and h.value is None
    assert "device" in bd.last_error()


def test_every_config_validates(toy):
    """All five workloads pass validation (the no-device error comes after it)."""
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    for fn in (wl.resnet20, wl.resnet50, wl.vgg16, wl.resnet101):
        s = fn()
        p = wl.gen_params(s, 1, True) if fn is wl.resnet20 else _light_params(s)
        c, hh, w = s.input_shape
        rc, _ = _create([s], [p], precision=bd.RAFIKI_BF16, opts_over={"c": c, "h": hh, "w": w})
        assert rc == bd.RAFIKI_ERR_HIP, (s.name, bd.last_error())
    s = wl.textcnn()
    rc, _ = _create([s], [_light_params(s)], precision=bd.RAFIKI_BF16,
                    opts_over={"input_kind": 1, "c": 1, "h": 256, "w": 1, "vocab": 30000})
    assert rc == bd.RAFIKI_ERR_HIP, bd.last_error()


def _light_params(spec):
    """Zero-filled parameters of the right shapes (validation only reads shapes)."""
    lp = []
    for L in spec.layers:
        p = wl.gen.LayerParams()
        if L.has_weight():
            p.weight = np.zeros(1, np.float32)
        if L.bias:
            p.bias = np.zeros(1, np.float32)
        if L.bn:
            p.bn_gamma = p.bn_beta = p.bn_mean = p.bn_var = np.zeros(1, np.float32)
        lp.append(p)
    return wl.ModelParams(spec, lp, 0, True)


def test_branch_fusion_keeps_validation_errors():
    """The bf16 pre-pass that fuses a TextCNN's branches reads the layer list before it
    is validated: malformed concatenations still fail validation, not the pre-pass."""
    import copy
    s = wl.textcnn(vocab=100, seq_len=16, dim=64, filters=8, widths=(2, 3, 4), n_classes=2)
    opts = {"input_kind": 1, "c": 1, "h": 16, "w": 1, "vocab": 100}
    # a concatenation whose c_out is not the sum of its inputs
    bad = copy.deepcopy(s)
    i = [k for k, L in enumerate(bad.layers) if L.op == wl.CONCAT][-1]
    bad.layers[i].c_out += 1
    rc, _ = _create([bad], [_light_params(bad)], precision=bd.RAFIKI_BF16, opts_over=opts)
    assert rc == bd.RAFIKI_ERR_INVALID and "concat" in bd.last_error()
    # a concatenation that reads a later layer
    bad = copy.deepcopy(s)
    i = [k for k, L in enumerate(bad.layers) if L.op == wl.CONCAT][0]
    bad.layers[i].input2 = len(bad.layers) - 1
    rc, _ = _create([bad], [_light_params(bad)], precision=bd.RAFIKI_BF16, opts_over=opts)
    assert rc == bd.RAFIKI_ERR_INVALID and "out of range" in bd.last_error()


def test_oversize_max_batch_rejected_at_create():
    """The bf16 GEMM addresses a layer's input through 32-bit offsets: VGG-16's
    224 x 224 x 64 activations exceed 2 GiB above about 334 requests.  create rejects
    such a max_batch before any device call (so no infer meets it partway); a
    max_batch just below the limit passes validation."""
    s = wl.vgg16()
    c, hh, w = s.input_shape
    opts = {"c": c, "h": hh, "w": w}
    rc, h = _create([s], [_light_params(s)], precision=bd.RAFIKI_BF16, max_batch=512, opts_over=opts)
    assert rc == bd.RAFIKI_ERR_UNSUPPORTED and h.value is None
    assert "max_batch" in bd.last_error() and "2 GiB" in bd.last_error()
    import torch
    if not torch.cuda.is_available():
        rc, _ = _create([s], [_light_params(s)], precision=bd.RAFIKI_BF16, max_batch=333, opts_over=opts)
        assert rc == bd.RAFIKI_ERR_HIP, bd.last_error()

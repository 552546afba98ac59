"""The Python binding's ctypes structures have the layout the C headers give the
structs (sizes and field offsets as compiled by the host C compiler), so no field is
misplaced across the boundary.  Needs gcc; no GPU."""
import ctypes as C
import os
import shutil
import subprocess

import pytest

from paper_1804_06087_amd import binding as bd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

STRUCTS = {
    "rafiki_layer": bd.RafikiLayer,
    "rafiki_model_desc": bd.RafikiModelDesc,
    "rafiki_ensemble_opts": bd.RafikiOpts,
    "rafiki_trace_rec": bd.RafikiTraceRec,
    "rafiki_greedy_policy": bd.RafikiGreedyPolicy,
    "rafiki_dispatch": bd.RafikiDispatch,
    "rafiki_rl_config": bd.RafikiRLConfig,
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_ctypes_layout_matches_headers(tmp_path):
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "rafiki_ensemble.h"',
             '#include "rafiki_sched.h"', '#include "rafiki_rl.h"', "int main(void) {"]
    for cname, py in STRUCTS.items():
        lines.append(f'  printf("{cname} size %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'  printf("{cname} {fname} %zu\\n", offsetof({cname}, {fname}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {}
    for line in out:
        if line:
            cname, field, val = line.split()
            got[(cname, field)] = int(val)
    for cname, py in STRUCTS.items():
        assert got[(cname, "size")] == C.sizeof(py), cname
        for fname, _ in py._fields_:
            assert got[(cname, fname)] == getattr(py, fname).offset, f"{cname}.{fname}"


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_binding_constants_match_headers(tmp_path):
    """Status codes, precisions and the direct-kernel tile id as the header defines them."""
    names = ["RAFIKI_OK", "RAFIKI_ERR_INVALID", "RAFIKI_ERR_UNSUPPORTED", "RAFIKI_ERR_NOMEM", "RAFIKI_ERR_HIP",
             "RAFIKI_FP32", "RAFIKI_BF16", "RAFIKI_TILE_DIRECT"]
    lines = ['#include <stdio.h>', '#include "rafiki_ensemble.h"', "int main(void) {"]
    lines += [f'  printf("{nm} %d\\n", (int)({nm}));' for nm in names]
    lines += ["  return 0;", "}"]
    src = tmp_path / "consts.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "consts"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = dict((ln.split()[0], int(ln.split()[1])) for ln in out if ln)
    for nm in names:
        assert got[nm] == getattr(bd, nm), nm

#!/usr/bin/env python3
"""Write the fp64 oracle's per-model logits of the configured request batches.

Every value in the files this script writes comes from ``oracle.run_model`` on the
seeded parameters and inputs of ``workloads``; nothing else is called.  The GPU
parity tests compare every row of a configured batch against these files instead
of re-running the oracle (about 17 minutes of CPU for the ImageNet-shaped batch).

Files (``numpy.savez_compressed``, float64 arrays ``<mode>_m<k>`` of shape
[rows, n_classes]; mode ``exact`` = fp64 throughout, ``bf16`` = every stored
inter-layer tensor rounded to bfloat16):

* ``oracle_logits_r50_vgg16_r101_n256.npz`` -- ResNet-50, VGG-16, ResNet-101 over
  the 256 ImageNet-shaped requests of the subset/batch-size sweep (the first 64 are
  the batch-64 workload);
* ``oracle_logits_resnet20x3_n128.npz`` -- three ResNet-20 over 128 CIFAR-shaped
  requests;
* ``oracle_logits_textcnn_x4_n512.npz`` -- four TextCNN over 512 token sequences.

Usage: ``python tests/golden/make_oracle_logits.py [imagenet|cifar|text ...]``
(default: all three).  Models run in parallel worker processes.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

FILES = {
    "imagenet": (4, "oracle_logits_r50_vgg16_r101_n256.npz", 2),
    "cifar": (2, "oracle_logits_resnet20x3_n128.npz", 16),
    "text": (5, "oracle_logits_textcnn_x4_n512.npz", 16),
}


def _one(cid: int, m: int, act, chunk: int):
    import oracle
    import workloads as wl
    cfg, specs, params, batch = wl.build_config(cid, models=[m])
    t = time.time()
    z = oracle.run_model(specs[0], params[0], batch, act=act, chunk=chunk)
    return m, act, z, time.time() - t


def make(which: str, workers: int) -> str:
    import workloads as wl
    cid, fname, chunk = FILES[which]
    n_models = len(wl.CONFIGS[cid].models)
    out = {}
    jobs = [(cid, m, act, chunk) for m in range(n_models) for act in (None, "bf16")]
    with cf.ProcessPoolExecutor(max_workers=min(workers, len(jobs))) as ex:
        for m, act, z, dt in ex.map(_one, *zip(*jobs)):
            key = f"{'bf16' if act else 'exact'}_m{m}"
            out[key] = np.asarray(z, np.float64)
            print(f"{which}: {key} {z.shape} in {dt:.0f} s", flush=True)
    path = os.path.join(HERE, fname)
    np.savez_compressed(path, **out)
    return path


def main(argv):
    which = argv[1:] or list(FILES)
    workers = int(os.environ.get("ORACLE_WORKERS", "3"))
    for w in which:
        print("wrote", make(w, workers), flush=True)


if __name__ == "__main__":
    main(sys.argv)

#!/usr/bin/env python3
"""Ensemble-inference benchmark on one MI355X.

A step is one call of the C ABI's infer over one request batch: input staging, the
forward pass of every selected model, and the combine.  Inputs and weights are
resident in HBM before timing starts.  Default workload: ResNet-50 + VGG-16 +
ResNet-101, batch 64 of 3x224x224 images, bf16 with fp32 accumulation, all three
models selected.

Prints ONE JSON line: throughput (images/s or sequences/s), ms per step, p50/p99
batch latency, the roofline of the dominant kernel class (timed live with HIP events
on the launch stream in a separate traced pass), and the fp64 CPU oracle timed on
a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "ensemble images/sec at batch 64 (bf16, 224²) + MFMA util %; p50 batch latency"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak
PEAK_FP32_TFLOPS = 157.3      # MI355X fp32 vector peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E

WORKLOADS = {
    # name: (config id, batch, mask, description)
    "c3": (3, 64, 0b111, "resnet50+vgg16+resnet101 ensemble, batch 64 of 3x224x224, bf16 (fp32 accumulate)"),
    "c2": (2, 128, 0b111, "3x resnet20 ensemble, batch 128 of 3x32x32, bf16 (fp32 accumulate)"),
    "c1": (1, 8, 0b11, "2x toy CNN ensemble, batch 8 of 3x32x32, fp32"),
    "c5": (5, 512, 0b1111, "4x textcnn ensemble, batch 512 of 256 tokens, bf16 (fp32 accumulate)"),
}


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="c3", choices=sorted(WORKLOADS) + ["c4"])
    ap.add_argument("--n", type=int, default=None, help="batch size (c4 sweep points, or override)")
    ap.add_argument("--mask", type=int, default=None, help="model subset mask override")
    ap.add_argument("--combine", default="mean", choices=["mean", "vote"],
                    help="ensemble combine: probability mean (default) or majority vote")
    ap.add_argument("--trace-steps", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target CPU time of the oracle sample")
    ap.add_argument("--pmc-copy-bytes", type=int, default=0,
                    help="after warmup, copy this many bytes with a plain device copy: under rocprofv3 --pmc it "
                         "calibrates FETCH_SIZE / WRITE_SIZE and marks where the measured steps begin")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of --pmc-copy-bytes into the "
                         "per-launch HBM traffic of the conv kernel and print it as JSON")
    ap.add_argument("--traffic-file", default=None, help="traffic JSON written by --summarize-pmc")
    ap.add_argument("--serve", default=None, choices=["sync", "async", "rl"],
                    help="instead of the step benchmark, serve a sine-rate request stream in real time with the "
                         "greedy batch-size policy: every batch through all selected models (sync) or each model "
                         "an independent server (async); prints one JSON line of serving statistics.  rl: profile "
                         "c(m, b) on the device, train the actor-critic subset/batch scheduler on it and compare "
                         "its policy with fixed policies in the simulated multi-model environment")
    ap.add_argument("--cycles", type=float, default=1.0, help="serving: sine cycles of 500 tau to serve")
    ap.add_argument("--period-taus", type=int, default=500, help="serving: sine period in units of tau")
    ap.add_argument("--rl-episodes", type=int, default=60, help="--serve rl: training episodes")
    ap.add_argument("--sweep", action="store_true",
                    help="latency/throughput trade-off of the ResNet-50 + VGG-16 + ResNet-101 subsets {R50}, "
                         "{R50, VGG-16}, {all} at batch sizes 1, 4, 16, 64, 256: one JSON line per point with "
                         "p50/p99 batch latency and images/s")
    ap.add_argument("--sweep-calls", type=int, default=200, help="sweep: timed calls per point")
    ap.add_argument("--memory-kernels", action="store_true",
                    help="HBM bandwidth of the path's memory-bound kernels called on their own (combine, vote, "
                         "max-pool, global average pool) at ImageNet-shaped sizes, against the 8 TB/s peak and a "
                         "plain device copy; one JSON line per kernel")
    ap.add_argument("--peaks", action="store_true",
                    help="the device's own ceilings: a register-resident bf16 MFMA loop (TFLOP/s) at 1, 2 and 4 "
                         "wavefronts per SIMD, a 4 GiB streaming read and a 2 GiB device copy (GB/s); one JSON "
                         "line each")
    ap.add_argument("--layers", action="store_true",
                    help="per-launch roofline of one workload (--workload, --n): traced steps with the models "
                         "one after another; for every launch its own bound max(FLOPs / 2.5 PFLOP/s, bytes / 8 TB/s) "
                         "and the fraction of it achieved; a markdown table")
    return ap.parse_args()


# the bf16 conv launches (trace class conv_mfma): the GEMM kernel and the direct conv kernel
CONV_SOURCES = [os.path.join(ROOT, "paper_1804_06087_amd", "csrc", f) for f in ("conv_mfma.hip", "conv_direct.hip")]
CONV_KERNEL_NAMES = ("conv_mfma_kernel", "conv_direct_kernel")


def strip_comments(src: str) -> str:
    """C++ source without its comments and blank space, so that editing a comment keeps
    the hash of the code (string literals in the kernel sources hold no comment marks)."""
    import re
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", "", src)
    return "\n".join(" ".join(line.split()) for line in src.splitlines() if line.strip())


def kernel_source_sha() -> str:
    """sha256 of the conv kernel sources' code (comments and layout ignored): the stored
    traffic counters are reported only while it matches."""
    import hashlib
    h = hashlib.sha256()
    for f in CONV_SOURCES:
        h.update(strip_comments(open(f).read()).encode())
    return h.hexdigest()


def _pmc_rows(d, counter):
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    rows = [r for r in csv.DictReader(open(files[0])) if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return [(r["Kernel_Name"], float(r["Counter_Value"]) * 1024.0) for r in rows]   # KiB -> bytes


def summarize_pmc(fetch_dir, write_dir, copy_bytes):
    """Per-launch HBM bytes of the conv kernel in the first traced pass (the models one
    after another: the launches whose average duration the roofline figure uses).

    bench.py runs the calibration copy just before and just after that pass.  FETCH_SIZE /
    WRITE_SIZE are in KiB per dispatch; each is rescaled by the ratio of the copy's known
    size to what the same counter read for the copy."""
    out = {}
    for name, d, counter in (("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")):
        rows = _pmc_rows(d, counter)
        # the copies: the largest dispatches that are not the library's (the buffer's
        # initial fill writes as much as a copy but reads nothing, and comes first)
        other = [i for i, (k, _) in enumerate(rows) if "rafiki" not in k]
        if not other:
            raise SystemExit(f"calibration copy not found in {d}")
        top = max(rows[i][1] for i in other)
        marks = [i for i in other if rows[i][1] >= 0.9 * top]
        if len(marks) < 2:
            raise SystemExit(f"the two marker copies around the traced pass were not found in {d}")
        a, b = marks[-2], marks[-1]
        c = b
        scale = copy_bytes / rows[c][1] if rows[c][1] > 0 else float("nan")
        conv = [v for k, v in rows[a + 1:b] if any(nm in k for nm in CONV_KERNEL_NAMES)]
        out[name] = {"scale": scale, "launches": len(conv), "bytes_per_launch": scale * sum(conv) / max(len(conv), 1),
                     "copy_counter_bytes": rows[c][1]}
    return {"kernel": "conv_mfma", "source_sha256": kernel_source_sha(), "copy_bytes": copy_bytes,
            "fetch": out["fetch"], "write": out["write"],
            "traffic_bytes_per_launch": out["fetch"]["bytes_per_launch"] + out["write"]["bytes_per_launch"]}


def cpu_baseline(specs, params, batch, mask, target_s, unit, combine="mean"):
    """Time the fp64 oracle (as is) on the host cores over a bounded sample of the batch."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    run = oracle.ensemble if combine == "mean" else oracle.ensemble_vote
    t0 = time.perf_counter()
    run(specs, params, batch[:1], mask)
    t1 = time.perf_counter() - t0
    k = int(max(1, min(batch.shape[0], round(target_s / max(t1, 1e-6)))))
    t0 = time.perf_counter()
    run(specs, params, batch[:k], mask)
    dt = time.perf_counter() - t0
    return {"value": round(k / dt, 4), "unit": unit, "cores": int(cores), "kind": "oracle",
            "sample": f"{k} of the {batch.shape[0]} requests, all selected models, fp64 NumPy oracle, "
                      f"{dt:.1f} s"}


def serve_main(args, dev):
    """Greedy serving experiment (Section 7.2) on one GPU: candidate sizes B = {16, 32,
    48, 64}, tau = 2 c(64), delta = 0.1 tau, sine arrivals with period 500 tau around the
    synchronous ensemble's throughput (sync) or the summed per-model throughput (async)."""
    import numpy as np
    import torch

    import oracle
    import workloads as wl
    from paper_1804_06087_amd import Ensemble

    cid = WORKLOADS[args.workload][0]
    mask = args.mask or WORKLOADS[args.workload][2]
    B = [16, 32, 48, 64]
    cfg, specs, params, pool = wl.build_config(cid, n=1024)
    C = specs[0].n_classes
    ens = Ensemble(specs, params, precision=cfg.precision, max_batch=max(B))
    xpool = torch.from_numpy(pool).to(dev)
    sel = [m for m in range(len(specs)) if (mask >> m) & 1]
    c_ens = ens.profile(xpool, B, mask, reps=10)
    c_mod = {m: ens.profile(xpool, B, 1 << m, reps=10) for m in sel}
    tau = int(2 * c_ens[-1])
    delta = tau // 10
    r_l = max(b / c for b, c in zip(B, c_ens)) * 1e6                       # all models on every batch
    r_u = sum(max(b / c for b, c in zip(B, c_mod[m])) * 1e6 for m in sel)  # each model its own server
    rate = r_l if args.serve == "sync" else r_u
    period = args.period_taus * tau
    arr = wl.sine_arrivals(rate, period, int(args.cycles * period), max(tau // 10, 1), seed=0)
    n = int(arr.size)
    req_bytes = n * xpool[0].numel() * xpool.element_size()
    if req_bytes > 48 * 2 ** 30:
        raise SystemExit(f"{n} requests need {req_bytes / 2 ** 30:.0f} GiB of HBM; lower --cycles or --period-taus")
    reps = (n + xpool.shape[0] - 1) // xpool.shape[0]
    x = xpool.repeat((reps,) + (1,) * (xpool.dim() - 1))[:n].contiguous()   # requests resident in HBM
    probs = torch.empty((n, C), dtype=torch.float32, device=dev)
    labels = torch.empty((n,), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if args.serve == "sync":
        lat, disp = ens.serve_greedy(x, arr, B, c_ens, tau, delta, mask, probs, labels, combine=args.combine)
    else:
        pols = {m: (B, c_mod[m], tau, delta) for m in sel}
        lat, disp = ens.serve_greedy_async(x, arr, pols, mask, probs, labels)
    wall = time.perf_counter() - t0
    # Equation (single) over the latencies the native loop measured: overdue requests
    # (latency above tau) and the mean exceeding time over all requests
    lat = np.asarray(lat, dtype=np.int64)
    served = lat[lat >= 0]
    st = {"requests": int(lat.size), "served": int(served.size), "overdue": int((served > tau).sum()),
          "mean_exceeding_us": float(np.maximum(served - tau, 0).sum() / max(lat.size, 1))}
    # the check, outside the timed region: the policy replayed by the scheduler oracle
    lat_sim = oracle.simulate_greedy(arr, B, dict(zip(B, c_ens.tolist())), tau, delta)[0] \
        if args.serve == "sync" else None
    dur_s = (int(disp["end_us"].max()) if len(disp) else 0) / 1e6
    out = {
        "metric": f"greedy serving, {'synchronous ensemble' if args.serve == 'sync' else 'asynchronous models'}: "
                  "overdue requests per second and mean exceeding time (Equation single)",
        "value": round(st["overdue"] / max(dur_s, 1e-9), 2), "unit": "overdue requests/s",
        "higher_is_better": False, "n_gpus": 1, "dtype": "bf16" if cfg.precision == "bf16" else "f32",
        "data": "synthetic requests (a 1024-image seeded pool tiled in HBM), seeded sine arrivals",
        "config": {"workload": WORKLOADS[args.workload][3], "mask": mask, "B": B, "tau_us": tau, "delta_us": delta,
                   "period_us": period, "arrival_ref_rate": round(rate, 1),
                   "arrival_ref": "r_l (synchronous ensemble throughput)" if args.serve == "sync"
                   else "r_u (sum of per-model throughputs)", "combine": args.combine if args.serve == "sync"
                   else "none (one model per batch)"},
        "c_b_us": {"ensemble": c_ens.tolist(), **{f"model{m}": c_mod[m].tolist() for m in sel}},
        "requests": st["requests"], "served": st["served"], "overdue": st["overdue"],
        "overdue_frac": round(st["overdue"] / max(st["requests"], 1), 4),
        "mean_exceeding_us": round(st["mean_exceeding_us"], 1),
        "latency_p50_us": int(np.percentile(served, 50)) if served.size else None,
        "latency_p99_us": int(np.percentile(served, 99)) if served.size else None,
        "served_per_s": round(st["served"] / max(dur_s, 1e-9), 1), "batches": int(len(disp)),
        "batch_sizes": {str(b): int((disp["b"] == b).sum()) for b in B},
        "wall_s": round(wall, 2),
    }
    if args.serve == "async":
        out["batches_per_model"] = {str(m): int((disp["model"] == m).sum()) for m in sel}
    if lat_sim is not None:
        so = oracle.serving_stats(lat_sim, tau)
        out["oracle_simulation"] = {"overdue": so["overdue"], "mean_exceeding_us": round(so["mean_exceeding_us"], 1),
                                    "served": so["served"],
                                    "note": "the policy replayed by the scheduler oracle with c(b) as profiled"}
    ens.close()
    print(json.dumps(out), flush=True)


def rl_main(args, dev):
    """Multi-model scheduling (Section 5.2): c(m, b) of each ImageNet-shaped model is
    profiled alone on the device (B = {16, 32, 48, 64}); the actor-critic agent is
    trained on sine arrivals in the simulated environment (each model an independent
    server); its policy (sampled, and its most probable action) is compared, on a fresh
    arrival draw, with fixed policies: every batch through all models, or through the
    fastest model only.  The
    accuracy table a(M[v]) is synthetic (no trained weights or labelled data)."""
    import numpy as np
    import torch

    import workloads as wl
    from paper_1804_06087_amd import Ensemble, RLScheduler

    B = [16, 32, 48, 64]
    cfg, specs, params, pool = wl.build_config(3, n=64)
    ens = Ensemble(specs, params, precision=cfg.precision, max_batch=max(B))
    x = torch.from_numpy(pool).to(dev)
    cost = np.stack([ens.profile(x, B, 1 << m, reps=10) for m in range(len(specs))]).astype(np.int64)
    ens.close()
    M = len(specs)
    base = [0.70, 0.71, 0.72]   # synthetic single-model accuracies, in model order
    acc = np.zeros(1 << M)
    for v in range(1, 1 << M):
        members = [m for m in range(M) if (v >> m) & 1]
        acc[v] = max(base[m] for m in members) + 0.015 * (len(members) - 1)
    tau = int(2 * cost[:, -1].max())
    r_all = max(b / cost[:, j].max() for j, b in enumerate(B)) * 1e6       # every batch through all models
    period = 50 * tau
    train_arr = wl.sine_arrivals(r_all, period, 3 * period, max(tau // 10, 1), seed=1)
    test_arr = wl.sine_arrivals(r_all, period, 3 * period, max(tau // 10, 1), seed=2)
    agent = RLScheduler(B, cost, acc, tau, 1.0, queue_features=64, hidden=64, seed=3)
    t0 = time.perf_counter()
    hist = agent.train(train_arr, episodes=args.rl_episodes, lr=3e-3, seed=4)
    train_s = time.perf_counter() - t0
    n_acts = agent.n_actions

    def evaluate(ep):
        lat = ep["latency"]
        served = lat >= 0
        acts = ep["actions"]
        sizes = [B[a % len(B)] for a in acts]
        masks = [a // len(B) + 1 for a in acts]
        return {"reward": round(float(ep["rewards"].sum()), 2),
                "reward_per_request": round(float(ep["rewards"].sum()) / max(lat.size, 1), 4),
                "served": int(served.sum()), "overdue": int((lat[served] > tau).sum()),
                "mean_accuracy_per_batch": round(float(np.mean([acc[m] for m in masks])) if masks else 0.0, 4),
                "decisions": int(len(acts)),
                "mask_counts": {str(v): int(sum(1 for m in masks if m == v)) for v in range(1, 1 << M)},
                "mean_requested_b": round(float(np.mean(sizes)) if sizes else 0.0, 1)}

    res = {"rl_sampled": evaluate(agent.run_episode(test_arr, mode="sample", seed=5)),
           "rl_argmax": evaluate(agent.run_episode(test_arr, mode="argmax"))}
    fixed = {"all_models_b64": (len(B) * ((1 << M) - 2) + len(B) - 1),
             "fastest_model_b64": None}
    fastest = int(np.argmin(cost[:, -1]))
    fixed["fastest_model_b64"] = ((1 << fastest) - 1) * len(B) + len(B) - 1
    for name, a in fixed.items():
        assert 0 <= a < n_acts
        res[name] = evaluate(agent.run_episode(test_arr, mode="given", actions=[a] * test_arr.size))
    out = {
        "metric": "RL subset/batch scheduler on the measured c(m, b): reward per request (Equation multi_acc_reward)",
        "value": res["rl_sampled"]["reward_per_request"], "unit": "reward/request", "higher_is_better": True,
        "n_gpus": 1, "dtype": "bf16",
        "data": "c(m, b) profiled on the device; seeded sine arrivals; synthetic accuracy table",
        "config": {"workload": WORKLOADS["c3"][3], "B": B, "tau_us": tau, "beta": 1.0, "period_us": period,
                   "arrival_ref_rate": round(r_all, 1), "accuracy_table": [round(a, 3) for a in acc.tolist()],
                   "episodes": args.rl_episodes, "requests_per_episode": int(train_arr.size)},
        "c_mb_us": cost.tolist(), "train_s": round(train_s, 2),
        "train_reward_first_last": [round(float(hist[:5].mean()), 2), round(float(hist[-5:].mean()), 2)],
        "policies": res,
    }
    print(json.dumps(out), flush=True)


def memory_main(args, dev):
    """Standalone memory-bound kernels: the combine at |S| = 3, C = 1000 on a scaled
    batch of 262,144 rows (the batch-64 combine moves about 1 MB, below launch latency),
    the ResNet stem max-pool at a scaled batch of 256 and the VGG-16 first max-pool at
    batch 64, and the global average pool of ResNet's last stage (batch 64 and a scaled
    batch of 2048); apart from the batch-64 pool, every working set exceeds the 256 MB
    last-level cache.  Each
    timing brackets enough back-to-back calls to last about a millisecond (so short
    kernels are not dominated by the events around them); best of 10 timings after 3
    warm-up calls; algorithmic bytes = every input and output once."""
    import torch

    from paper_1804_06087_amd.binding import (combine_mean, combine_vote, maxpool_nhwc_bf16,
                                              global_avgpool_nhwc_bf16)

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        reps = 1
        best = 1e30
        for i in range(11):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(reps):
                fn()
            b.record()
            b.synchronize()
            ms = a.elapsed_time(b) / reps
            if i == 0:      # sizing run
                reps = max(1, min(200, int(1.0 / max(ms, 1e-3))))
                continue
            best = min(best, ms)
        return best

    def emit(name, shape, nbytes, ms):
        gbs = nbytes / (ms / 1e3) / 1e9
        print(json.dumps({"metric": f"HBM bandwidth of {name}", "value": round(gbs, 1), "unit": "GB/s",
                          "higher_is_better": True, "n_gpus": 1, "dtype": "f32" if "combine" in name or "vote" in name
                          else "bf16", "data": "synthetic", "config": {"kernel": name, "shape": shape},
                          "ms": round(ms, 4), "bytes": int(nbytes),
                          "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                                       "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)}}), flush=True)

    g = torch.Generator(device=dev)
    g.manual_seed(0)
    # plain device copy, for context (read + write)
    src = torch.empty(2 ** 28, dtype=torch.float32, device=dev).normal_(generator=g)
    dst = torch.empty_like(src)
    emit("device copy (torch)", [2 ** 28], 2 * src.numel() * 4, timed(lambda: dst.copy_(src)))
    del src, dst
    S, n, C = 3, 262144, 1000
    z = torch.empty((S, n, C), dtype=torch.float32, device=dev).normal_(generator=g)
    p = torch.empty((n, C), dtype=torch.float32, device=dev)
    lab = torch.empty((n,), dtype=torch.int32, device=dev)
    nb = n * C * 4 * (S + 1) + 4 * n
    emit("combine (softmax, mean, argmax)", [S, n, C], nb, timed(lambda: combine_mean(z, p, lab)))
    emit("majority-vote combine", [S, n, C], nb, timed(lambda: combine_vote(z, p, lab)))
    del z, p, lab
    # Every benchmarked working set exceeds the 256 MB last-level cache (MALL), so that the
    # algorithmic bytes of back-to-back calls are HBM bytes.
    for name, (N, H, W, Cc), k, st, pd in (("max-pool 3x3/2 pad 1 (ResNet stem)", (256, 112, 112, 64), 3, 2, 1),
                                         ("max-pool 2x2/2 (VGG-16 pool1)", (64, 224, 224, 64), 2, 2, 0)):
        x = torch.empty((N, H, W, Cc), dtype=torch.bfloat16, device=dev).normal_(generator=g)
        Ho, Wo = (H + 2 * pd - k) // st + 1, (W + 2 * pd - k) // st + 1
        y = torch.empty((N, Ho, Wo, Cc), dtype=torch.bfloat16, device=dev)
        emit(name, [N, H, W, Cc], (x.numel() + y.numel()) * 2, timed(lambda: maxpool_nhwc_bf16(x, y, k, st, pd)))
        del x, y
    for N in (64, 2048):    # batch 64 as configured (13 MB: launch-bound), and a scaled batch
        x = torch.empty((N, 7, 7, 2048), dtype=torch.bfloat16, device=dev).normal_(generator=g)
        y = torch.empty((N, 2048), dtype=torch.bfloat16, device=dev)
        emit("global average pool (ResNet last stage)", [N, 7, 7, 2048], (x.numel() + y.numel()) * 2,
             timed(lambda: global_avgpool_nhwc_bf16(x, y)))
        del x, y


def peaks_main(args, dev):
    """Measured ceilings of this MI355X: the kernels' rooflines use the published peaks
    (2.5 PFLOP/s bf16 dense, 8 TB/s); these probes show what the device delivers to a
    kernel that does nothing else.  MFMA: 256 workgroups x 4 wavefronts per pass over the
    256 compute units (1, 2 or 4 wavefronts per SIMD), each wavefront 8 independent
    32x32x16 bf16 MFMAs per iteration on register operands.  HBM: one 16-byte streaming
    read pass over 4 GiB (16x the last-level cache), and a device-to-device copy of
    2 GiB (read + write).  Main-loop skeleton: the GEMM kernel's LDS fragment reads and
    MFMAs for four wave layouts, alone and with each K tile's LDS writes and barrier, one
    workgroup per compute unit.  Best of 10 (skeleton: 5) timings after 2 warm-ups, HIP
    events."""
    import torch

    from paper_1804_06087_amd.binding import probe_mfma_bf16, probe_hbm_read

    def best_ms(fn, reps=10):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        t = 1e30
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            b.synchronize()
            t = min(t, a.elapsed_time(b))
        return t

    def emit(name, value, unit, peak, cfg, ms):
        print(json.dumps({"metric": f"measured ceiling: {name}", "value": round(value, 1), "unit": unit,
                          "higher_is_better": True, "n_gpus": 1, "dtype": "bf16" if "MFMA" in name else "u8",
                          "data": "synthetic", "config": cfg, "ms": round(ms, 4),
                          "of_published_peak": round(value / peak, 4), "published_peak": peak}), flush=True)

    iters = 20000
    for per_simd in (1, 2, 4):
        blocks = 256 * per_simd
        out = torch.empty(blocks * 4, dtype=torch.float32, device=dev)
        ms = best_ms(lambda: probe_mfma_bf16(blocks, iters, out))
        flops = blocks * 4 * iters * 8 * 32768.0
        emit("register-resident bf16 MFMA loop", flops / (ms / 1e3) / 1e12, "TFLOP/s", PEAK_BF16_TFLOPS,
             {"kernel": "v_mfma_f32_32x32x16_bf16", "workgroups": blocks, "waves_per_simd": per_simd,
              "iterations": iters}, ms)
    # the GEMM kernel's main loop without memory loads (one workgroup per compute unit)
    from paper_1804_06087_amd.binding import MAINLOOP_VARIANTS, probe_mainloop
    ktiles, blocks = 2000, 256
    out = torch.empty(blocks * 8, dtype=torch.float32, device=dev)
    for variant, (waves, wtile, tile, mf) in MAINLOOP_VARIANTS.items():
        for sync in (False, True):
            ms = best_ms(lambda: probe_mainloop(variant, sync, blocks, ktiles, out), reps=5)
            flops = blocks * waves * ktiles * 4 * mf * 32768.0
            emit("GEMM main-loop skeleton (LDS fragment reads + MFMA" + (", tile writes + barrier" if sync else "") + ")",
                 flops / (ms / 1e3) / 1e12, "TFLOP/s", PEAK_BF16_TFLOPS,
                 {"kernel": "probe_mainloop", "waves": waves, "wave_tile": wtile, "workgroup_tile": tile,
                  "k_tiles": ktiles, "workgroups": blocks, "lds_writes_and_barrier_per_k_tile": sync}, ms)
    nbytes = 4 << 30
    x = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    x.fill_(7)
    blocks = 256 * 8
    out = torch.empty(blocks * 4, dtype=torch.int32, device=dev)
    ms = best_ms(lambda: probe_hbm_read(x, blocks, out))
    emit("HBM streaming read", nbytes / (ms / 1e3) / 1e9, "GB/s", PEAK_HBM_GBS,
         {"kernel": "16-byte nontemporal loads", "bytes": nbytes, "workgroups": blocks}, ms)
    del x
    src = torch.empty(1 << 29, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    ms = best_ms(lambda: dst.copy_(src))
    emit("device copy (read + write)", 2 * src.numel() * 4 / (ms / 1e3) / 1e9, "GB/s", PEAK_HBM_GBS,
         {"kernel": "torch copy_", "bytes_read": src.numel() * 4, "bytes_written": src.numel() * 4}, ms)


def sweep_cpu_baseline(specs, params, pool, n, mask):
    """The fp64 oracle (as is) over the first n requests and the selected models: one
    timed run after a one-request warm-up; images/s on the host cores."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    oracle.ensemble(specs, params, pool[:1], mask)
    t0 = time.perf_counter()
    oracle.ensemble(specs, params, pool[:n], mask)
    dt = time.perf_counter() - t0
    return {"value": round(n / dt, 4), "unit": "images/s", "cores": int(cores), "kind": "oracle",
            "sample": f"all {n} requests of the point, selected models, fp64 NumPy oracle, one run of {dt:.1f} s"}


def sweep_main(args, dev):
    """Latency/accuracy trade-off grid (Section 5.2): every subset of the ImageNet-shaped
    ensemble at every batch size, one handle (max batch 256) over one 256-image draw whose
    prefixes are the batches.  Per point: 20 warm-up calls, then timed calls each bracketed
    by events on the launch stream and synchronised; p50/p99 latency, images/s = n / p50.
    At n <= 4 also the cold latency: before each of 50 timed calls a 1 GiB buffer is
    written (outside the events), which evicts the weights from the last-level cache.
    Roofline per point: the algorithmic FLOPs and bytes of the call's launches (from one
    traced call) against p50 -- the MFMA fraction, and the fraction of the sum of the
    launches' own bounds max(FLOPs / 2.5 PFLOP/s, bytes / 8 TB/s).  CPU baseline at n =
    1, 16 and 64: the fp64 oracle over the same n requests and subset, timed once after
    a one-request warm-up (the n <= 64 points only; nothing is extrapolated)."""
    import numpy as np
    import torch

    import workloads as wl
    from paper_1804_06087_amd import Ensemble

    cfg, specs, params, pool = wl.build_config(4)
    C = specs[0].n_classes
    ens = Ensemble(specs, params, precision=cfg.precision, max_batch=max(cfg.batches))
    xpool = torch.from_numpy(pool).to(dev)
    probs = torch.empty((max(cfg.batches), C), dtype=torch.float32, device=dev)
    labels = torch.empty((max(cfg.batches),), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    names = ["resnet50", "vgg16", "resnet101"]
    flush = torch.empty(2 ** 28, dtype=torch.float32, device=dev)   # 1 GiB
    for mask in cfg.masks:
        for n in cfg.batches:
            x = xpool[:n]
            for _ in range(20):
                ens.infer(x, n, mask, probs, labels, stream)
            torch.cuda.synchronize()
            lat = []
            t_end = time.perf_counter() + 1.0
            while len(lat) < args.sweep_calls or time.perf_counter() < t_end:
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record(stream)
                ens.infer(x, n, mask, probs, labels, stream)
                b.record(stream)
                b.synchronize()
                lat.append(a.elapsed_time(b))
            lat = np.array(lat)
            p50 = float(np.percentile(lat, 50))
            # algorithmic work of one call (launches traced one after another)
            ens.trace(True)
            ens.infer(x, n, mask, probs, labels, stream)
            torch.cuda.synchronize()
            recs = ens.trace_read()
            ens.trace(False)
            flops = sum(r["flops"] for r in recs)
            nbytes = sum(r["bytes"] for r in recs)
            bound_ms = sum(max(r["flops"] / (PEAK_BF16_TFLOPS * 1e9), r["bytes"] / (PEAK_HBM_GBS * 1e6))
                           for r in recs)
            tflops = flops / (p50 / 1e3) / 1e12
            roof = {"bound": "mfma" if flops / (PEAK_BF16_TFLOPS * 1e9) >= nbytes / (PEAK_HBM_GBS * 1e6) else "hbm",
                    "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                    "frac": round(tflops / PEAK_BF16_TFLOPS, 4), "alg_gflop": round(flops / 1e9, 2),
                    "alg_gbytes": round(nbytes / 1e9, 3), "of_launch_roofline": round(bound_ms / p50, 4)}
            cpu = None
            if n in (1, 16, 64) and not args.no_cpu_baseline:
                cpu = sweep_cpu_baseline(specs, params, pool, n, mask)
            cold = None
            if n <= 4:
                cl = []
                for _ in range(50):
                    flush.fill_(1.0)
                    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    a.record(stream)
                    ens.infer(x, n, mask, probs, labels, stream)
                    b.record(stream)
                    b.synchronize()
                    cl.append(a.elapsed_time(b))
                cold = {"p50_ms": round(float(np.percentile(cl, 50)), 4),
                        "p99_ms": round(float(np.percentile(cl, 99)), 4), "calls": len(cl)}
            print(json.dumps({
                "metric": "ensemble images/sec and batch latency, subset/batch-size sweep",
                "value": round(n / (p50 / 1e3), 2), "unit": "images/s", "n_gpus": 1, "higher_is_better": True,
                "dtype": "bf16", "data": "synthetic (seeded N(0,1) images rounded to bf16, random-init weights)",
                "config": {"workload": "+".join(names[m] for m in range(3) if (mask >> m) & 1)
                           + f", batch {n} of 3x224x224", "mask": mask, "global_batch": n,
                           "schedule": schedule_desc(ens, n, mask, names)},
                "p50_ms": round(p50, 4), "p99_ms": round(float(np.percentile(lat, 99)), 4),
                "calls": int(lat.size), "cold": cold, "roofline": roof, "cpu_baseline": cpu}), flush=True)
    del flush
    ens.close()


def layers_main(args, dev):
    """Per-launch roofline table of one workload: every launch of three traced steps
    (models one after another, each kernel alone on the GPU), averaged per (model,
    layer, kernel class).  A launch's bound is max(FLOPs / bf16 peak, bytes / HBM peak)
    with its algorithmic FLOPs and bytes; 'of bound' = that time / measured time."""
    import numpy as np
    import torch

    import workloads as wl
    from workloads.specs import OP_NAMES
    from paper_1804_06087_amd import Ensemble

    cid = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5}[args.workload]
    cfg, specs, params, batch = wl.build_config(cid, n=args.n)
    n = batch.shape[0]
    mask = args.mask or (1 << len(specs)) - 1
    C = specs[0].n_classes
    ens = Ensemble(specs, params, precision=cfg.precision, max_batch=n)
    x = torch.from_numpy(batch).to(dev)
    probs = torch.empty((n, C), dtype=torch.float32, device=dev)
    labels = torch.empty((n,), dtype=torch.int32, device=dev)
    for _ in range(3):
        ens.infer(x, n, mask, probs, labels)
    torch.cuda.synchronize()
    ens.trace(True)
    T = 3
    for _ in range(T):
        ens.infer(x, n, mask, probs, labels)
    recs = ens.trace_read()
    ens.trace(False)
    ens.close()
    agg = {}
    for r in recs:
        key = (r["model"], r["layer"], r["kind"])
        a = agg.setdefault(key, {"ms": 0.0, "flops": r["flops"], "bytes": r["bytes"], "cfg": r["tile_cfg"],
                                 "splits": r["splits"]})
        a["ms"] += r["ms"] / T
    tot_ms = sum(a["ms"] for a in agg.values())
    tot_bound = 0.0
    from paper_1804_06087_amd.binding import tile_configs
    n_gemm_cfgs = len(tile_configs())   # the trace's tile id of the direct conv kernel
    print(f"# Per-launch roofline: {cfg.name}, batch {n}, mask {mask:#b}\n")
    print(f"Command: `python bench.py --layers --workload {args.workload}"
          + (f" --n {args.n}" if args.n else "") + (f" --mask {args.mask}" if args.mask else "") + "`\n")
    print("| model | layer | op | kernel | tile / splits | us | TFLOP/s | GB/s | bound | bound us | of bound |")
    print("|---|---|---|---|---|---|---|---|---|---|---|")
    by_kind = {}
    for (m, li, kind), a in sorted(agg.items(), key=lambda t: (t[0][0], t[0][1])):
        t_f = a["flops"] / (PEAK_BF16_TFLOPS * 1e12) * 1e3
        t_b = a["bytes"] / (PEAK_HBM_GBS * 1e9) * 1e3
        bound, tb = ("mfma", t_f) if t_f >= t_b else ("hbm", t_b)
        tot_bound += tb
        k = by_kind.setdefault(kind, [0.0, 0.0])
        k[0] += a["ms"]
        k[1] += tb
        desc = ""
        if m >= 0 and li >= 0:
            L = specs[m].layers[li]
            desc = f"{OP_NAMES[L.op]} {L.c_in}->{L.c_out} {L.kh}x{L.kw}/{L.stride}"
            if OP_NAMES[L.op] == "concat" and kind != "concat":   # branches fused into one GEMM + max
                desc = f"conv1d_maxtime branches -> concat {L.c_out}"
        tile = ("direct" if a["cfg"] == n_gemm_cfgs else f"{a['cfg']} / {a['splits']}") if a["cfg"] >= 0 else ""
        print(f"| {specs[m].name if m >= 0 else '-'} | {li} | {desc} | {kind} | {tile} | {a['ms'] * 1e3:.1f} | "
              f"{a['flops'] / a['ms'] / 1e9:.0f} | {a['bytes'] / a['ms'] / 1e6:.0f} | {bound} | {tb * 1e3:.1f} | "
              f"{tb / a['ms']:.2f} |")
    print(f"\nTotal traced time {tot_ms:.3f} ms per step; sum of the launches' roofline times {tot_bound:.3f} ms "
          f"({tot_bound / tot_ms:.3f} of the measured time).\n")
    print("| kernel class | ms per step | roofline ms | of bound |\n|---|---|---|---|")
    for kind, (ms, tb) in sorted(by_kind.items(), key=lambda t: -t[1][0]):
        print(f"| {kind} | {ms:.3f} | {tb:.3f} | {tb / ms:.2f} |")


def schedule_desc(ens, n, mask, names, kinds=()):
    """How the selected models' forward passes were scheduled for (n, mask); `kinds`
    are the kernel classes a traced pass launched."""
    members = [m for m in range(len(names)) if (mask >> m) & 1]
    if "fused_net" in kinds:
        return (f"whole-network kernel: one launch for the {len(members)} selected models, one workgroup per "
                "image and model, activations in LDS")
    if len(members) == 1:
        return names[members[0]]
    kinds = {names[m].split("#")[0] for m in members}
    if len(kinds) == 1 and os.environ.get("RAFIKI_GROUPED", "1") != "0":
        return f"grouped: one launch per layer for the {len(members)} {kinds.pop()} members"
    try:
        solo, asc = ens.get_schedule(n, mask)
        pa, pb = ens.get_schedule_pair(n, mask)
        lean = ens.get_schedule_tiles(n, mask)
    except Exception:
        solo, asc, pa, pb, lean = -1, 0, -1, -1, 0
    tiles = "; the layers of maps up to 14x14 on their lean tiles" if lean else ""
    if lean == 2 and solo >= 0:
        tiles += f", {names[solo]}'s direct-conv layers on GEMM tiles"
    if pa >= 0:
        rest = [names[m] for m in members if m not in (pa, pb)]
        return (f"{names[pa]} and {names[pb]} paired on one lane; {', '.join(rest) or 'nothing'} on a second lane"
                + tiles)
    if solo < 0:
        return "all concurrent" + tiles
    rest = [names[m] for m in members if m != solo]
    order = "shortest" if asc else "longest"
    return (f"{names[solo]} alone; {', '.join(rest)} one after another on a second lane, {order} alone time first"
            + tiles)


def main():
    args = parse()
    if args.summarize_pmc:
        if not args.pmc_copy_bytes:
            raise SystemExit("--summarize-pmc needs --pmc-copy-bytes (the calibration copy's size)")
        print(json.dumps(summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.pmc_copy_bytes)))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1 "
                                   "(sharding is described in the design notes, not implemented)"}))
        sys.exit(2)

    import numpy as np
    import torch

    import workloads as wl
    from paper_1804_06087_amd import Ensemble

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    dev = torch.device("cuda:0")
    if args.serve == "rl":
        rl_main(args, dev)
        return
    if args.serve:
        serve_main(args, dev)
        return
    if args.sweep:
        sweep_main(args, dev)
        return
    if args.memory_kernels:
        memory_main(args, dev)
        return
    if args.peaks:
        peaks_main(args, dev)
        return
    if args.layers:
        layers_main(args, dev)
        return

    if args.workload == "c4":
        cid, n, mask, desc = 4, args.n or 64, args.mask or 0b111, None
        desc = f"resnet50+vgg16+resnet101 subset mask {mask:#05b}, batch {n} of 3x224x224, bf16 (fp32 accumulate)"
    else:
        cid, n, mask, desc = WORKLOADS[args.workload]
        if args.n:
            n = args.n
        if args.mask:
            mask = args.mask
    cfg, specs, params, batch = wl.build_config(cid, n=n)
    precision = cfg.precision
    tokens = cfg.input_dist == "tokens"
    unit = "sequences/s" if tokens else "images/s"
    C = specs[0].n_classes

    ens = Ensemble(specs, params, precision=precision, max_batch=n)
    x = torch.from_numpy(batch).to(dev)
    probs = torch.empty((n, C), dtype=torch.float32, device=dev)
    labels = torch.empty((n,), dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()
    serve = ens.infer if args.combine == "mean" else ens.infer_vote

    for _ in range(args.warmup):
        serve(x, n, mask, probs, labels, stream)
    torch.cuda.synchronize()
    if args.pmc_copy_bytes:
        # a plain elementwise kernel that reads and writes pmc_copy_bytes each: it calibrates
        # the counters, and its two runs around the first traced pass mark the launches measured
        pmc_src = torch.empty(args.pmc_copy_bytes // 4, dtype=torch.float32, device=dev).fill_(1.0)
        pmc_dst = torch.empty_like(pmc_src)
        torch.cuda.synchronize()

    def pmc_mark():
        if args.pmc_copy_bytes:
            torch.cuda.synchronize()
            torch.mul(pmc_src, 1.0, out=pmc_dst)
            torch.cuda.synchronize()

    # ---- throughput: K back-to-back steps bracketed by synchronisation
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record(stream)
    for _ in range(args.steps):
        serve(x, n, mask, probs, labels, stream)
    ev1.record(stream)
    torch.cuda.synchronize()
    ms_per_step = ev0.elapsed_time(ev1) / args.steps

    # ---- host cost of enqueueing one step (device idle, no synchronisation inside)
    host = []
    for _ in range(5):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        serve(x, n, mask, probs, labels, stream)
        host.append((time.perf_counter() - t0) * 1e3)
    torch.cuda.synchronize()

    # ---- latency: each step on its own, events on the launch stream
    lat = []
    for _ in range(max(args.steps, 10)):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        serve(x, n, mask, probs, labels, stream)
        b.record(stream)
        b.synchronize()
        lat.append(a.elapsed_time(b))
    lat = np.array(lat)

    # ---- traced pass: per-launch HIP events around every kernel (separate from the timed steps)
    pmc_mark()
    ens.trace(True)
    for _ in range(args.trace_steps):
        serve(x, n, mask, probs, labels, stream)
    recs = ens.trace_read()
    ens.trace(False)
    torch.cuda.synchronize()
    pmc_mark()
    classes = {}
    flop_peak = (PEAK_BF16_TFLOPS if precision == "bf16" else PEAK_FP32_TFLOPS) * 1e12
    for r in recs:
        c = classes.setdefault(r["kind"], {"launches": 0, "ms": 0.0, "flops": 0.0, "bytes": 0.0, "bound_ms": 0.0})
        c["launches"] += 1
        c["ms"] += r["ms"]
        c["flops"] += r["flops"]
        c["bytes"] += r["bytes"]
        # this launch's own roofline time: the larger of its FLOPs at peak and its bytes at peak
        c["bound_ms"] += max(r["flops"] / flop_peak, r["bytes"] / (PEAK_HBM_GBS * 1e9)) * 1e3
    traced_step_ms = sum(c["ms"] for c in classes.values()) / args.trace_steps
    kernels = {}
    for k, c in classes.items():
        ent = {"launches_per_step": c["launches"] // args.trace_steps, "ms_per_step": round(c["ms"] / args.trace_steps, 4),
               "share": round(c["ms"] / args.trace_steps / traced_step_ms, 4)}
        if c["flops"] > 0:
            ent["tflops"] = round(c["flops"] / c["ms"] / 1e9, 2)
        ent["gbs_alg"] = round(c["bytes"] / c["ms"] / 1e6, 1)
        # time-weighted fraction of the per-launch roofline (each launch against its own bound)
        ent["of_launch_roofline"] = round(c["bound_ms"] / c["ms"], 4)
        kernels[k] = ent
    dom = max(classes, key=lambda k: classes[k]["ms"])
    d = classes[dom]
    if d["flops"] > 0:
        peak = PEAK_BF16_TFLOPS if precision == "bf16" else PEAK_FP32_TFLOPS
        achieved = d["flops"] / d["ms"] / 1e9
        roof = {"bound": "mfma" if precision == "bf16" else "alu", "achieved": round(achieved, 2), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4), "traffic": None,
                "kernel": dom, "avg_launch_ms": round(d["ms"] / d["launches"], 5),
                "alg_flops_per_launch": round(d["flops"] / d["launches"], 1)}
    else:
        achieved = d["bytes"] / d["ms"] / 1e6
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None, "kernel": dom,
                "avg_launch_ms": round(d["ms"] / d["launches"], 5),
                "alg_bytes_per_launch": round(d["bytes"] / d["launches"], 1)}

    # The same kernel class timed inside steps that keep the timed schedule (models on
    # their own streams): each launch then shares the GPU with the other lane, so its
    # duration includes waiting for compute units; reported beside the figure above.
    if len(specs) > 1:
        ens.trace(True, concurrent=True)
        for _ in range(args.trace_steps):
            serve(x, n, mask, probs, labels, stream)
        crecs = [r for r in ens.trace_read() if r["kind"] == dom]
        ens.trace(False)
        torch.cuda.synchronize()
        if crecs:
            cms = sum(r["ms"] for r in crecs) / len(crecs)
            roof["concurrent_avg_launch_ms"] = round(cms, 5)
            per_launch = d["flops"] / d["launches"] if d["flops"] > 0 else d["bytes"] / d["launches"]
            roof["concurrent_achieved"] = round(per_launch / cms / (1e9 if d["flops"] > 0 else 1e6), 2)

    # HBM traffic of the dominant kernel from committed counter runs, if they were
    # taken on the current kernel source
    traffic_names = {"c3": "r50_vgg16_r101_b64"}   # workloads whose conv traffic counters are committed
    tfile = args.traffic_file or (os.path.join(ROOT, "profiles", f"conv_mfma_traffic_{traffic_names[args.workload]}.json")
                                  if args.workload in traffic_names else "")
    if dom == "conv_mfma" and os.path.exists(tfile):
        try:
            t = json.load(open(tfile))
            if t.get("source_sha256") == kernel_source_sha():
                roof["traffic"] = round(t["traffic_bytes_per_launch"], 1)
                roof["traffic_unit"] = "bytes per launch (HBM, counter-based)"
        except Exception:
            pass
    step_flops = sum(c["flops"] for c in classes.values()) / args.trace_steps
    value = n / (ms_per_step / 1e3)
    out = {
        "metric": METRIC if args.workload == "c3" and args.combine == "mean" else
        f"ensemble {unit} ({args.workload}, majority vote)" if args.combine == "vote" else f"ensemble {unit} ({args.workload})",
        "value": round(value, 2),
        "unit": unit,
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if precision == "bf16" else "f32",
        "data": "synthetic (seeded inputs and random-init weights of the named architectures)",
        "config": {"workload": desc, "global_batch": n, "mask": mask, "n_classes": C, "combine": args.combine,
                   "input": "int32 tokens [n, 256]" if tokens else "float32 NCHW images",
                   "schedule": schedule_desc(ens, n, mask, [f"{sp.name}#{i}" for i, sp in enumerate(specs)],
                                             tuple(classes))},
        "p50_ms": round(float(np.percentile(lat, 50)), 4),
        "p99_ms": round(float(np.percentile(lat, 99)), 4),
        "host_enqueue_ms": round(float(np.median(host)), 4),
        "mfma_util_step": round(step_flops / (ms_per_step / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4)
        if precision == "bf16" else None,
        "alg_tflop_per_step": round(step_flops / 1e12, 4),
        "roofline": roof,
        "kernels": kernels,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(specs, params, batch, mask, args.cpu_seconds, unit,
                                        args.combine)
    ens.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

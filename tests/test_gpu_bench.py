"""bench.py on the device: one short run of the ResNet-20 x 3 workload prints one JSON
line with the fields of the benchmark contract (throughput, timing, roofline of the
dominant kernel with its live launch time, the CPU-oracle baseline)."""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402

pytestmark = pytest.mark.gpu


def test_bench_line_has_the_contract_fields(monkeypatch, capsys):
    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", "c2", "--steps", "3", "--warmup", "1",
                                      "--trace-steps", "1", "--cpu-seconds", "0.3"])
    bench.main()
    lines = [l for l in capsys.readouterr().out.splitlines() if l.startswith("{")]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1 and d["value"] > 0
    assert abs(d["value"] - d["config"]["global_batch"] / (d["ms_per_step"] / 1e3)) / d["value"] < 1e-3
    r = d["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in r, k
    assert r["bound"] == "mfma" and r["peak"] == 2500.0 and 0 < r["frac"] < 1
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-3
    # the same kernel timed in the concurrent schedule (three models): a longer launch
    assert r["concurrent_avg_launch_ms"] > 0 and r["concurrent_achieved"] > 0
    c = d["cpu_baseline"]
    assert c["kind"] == "oracle" and c["value"] > 0 and c["cores"] >= 1
    for kind in d["kernels"].values():
        assert kind["of_launch_roofline"] > 0   # can exceed 1 when a launch's data comes from cache

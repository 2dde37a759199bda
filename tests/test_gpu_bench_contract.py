"""bench.py's output line on the GPU: one JSON object with the fields the benchmark
reports (throughput, roofline entry, CPU baseline), on the tiny workload so that the
run and its CPU oracle take seconds."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_prints_one_complete_json_line():
    cmd = [sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--steps", "5", "--warmup", "2",
           "--settle-s", "0.05", "--no-variants"]
    print("[bench-contract] " + " ".join(cmd[1:]), flush=True)
    res = subprocess.run(cmd, cwd=ROOT, capture_output=True, text=True, timeout=240)
    assert res.returncode == 0, res.stderr[-2000:]
    lines = [ln for ln in res.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1, res.stdout
    r = json.loads(lines[0])
    for k, t in (("metric", str), ("value", float), ("unit", str), ("n_gpus", int), ("steps", int),
                 ("warmup", int), ("ms_per_step", float), ("higher_is_better", bool), ("scaling", str),
                 ("dtype", str), ("data", str), ("config", dict), ("roofline", dict), ("cpu_baseline", dict)):
        assert isinstance(r.get(k), t), (k, r.get(k))
    assert r["n_gpus"] == 1 and r["steps"] == 5 and r["warmup"] == 2 and r["vs_baseline"] is None
    assert r["value"] > 0 and r["ms_per_step"] > 0 and r["higher_is_better"] is True
    assert r["config"]["workload"].startswith("tiny:")
    rf = r["roofline"]
    assert rf["bound"] == "mfma" and rf["unit"] == "TOP/s" and rf["peak"] == 5000.0
    assert 0 < rf["achieved"] < rf["peak"] and abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-4
    assert rf["kernel_us"] > 0
    cb = r["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and "bit-exact vs GPU: True" in cb["sample"]
    assert cb["single_thread"]["tops"] > 0 and cb["single_thread"]["cores"] == 1
    assert r["settle"]["steps"] >= 1

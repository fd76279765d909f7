"""The benchmark's output contract: one JSON line with the fields the
measurement needs (metric, value, unit, timing, roofline, CPU baseline), and
a clear refusal to run on more than one GPU."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.gpu
def test_json_line_fields():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print("case bench contract: tiny workload, 2 steps", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "tiny", "--steps", "2",
                        "--warmup", "1", "--cpu-budget", "1"], capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k, t in [("metric", str), ("value", float), ("unit", str), ("n_gpus", int), ("steps", int),
                 ("warmup", int), ("ms_per_step", float), ("higher_is_better", bool), ("scaling", str),
                 ("dtype", str), ("data", str), ("config", dict), ("roofline", dict), ("cpu_baseline", dict)]:
        assert isinstance(d[k], t), (k, d.get(k))
    assert "vs_baseline" in d and d["vs_baseline"] is None
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1 and d["value"] > 0
    assert d["settle"]["slept_s"] >= 0 and d["settle"]["since_start_s"] + d["settle"]["slept_s"] >= 3.0 - 1e-3
    assert d["config"]["workload"].startswith("tiny")
    roof = d["roofline"]
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-3 and "traffic" in roof
    seeds = [x["seed"] for x in d["per_seed"]]
    assert seeds == [0, 1, 2] and d["config"]["seeds"] == [0, 1, 2]
    assert all(x["frac"] > 0 and x["mean_us"] > 0 for x in d["per_seed"])
    assert d["median_over_seeds"]["frac"] == sorted(x["frac"] for x in d["per_seed"])[1]
    ce = d["ceiling"]
    assert ce["copy_GBps"] > 0 and ce["gather_GBps"] > 0 and ce["pack_over_gather"] > 0
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["cores"] == 1 and cb["value"] > 0 and cb["unit"] and cb["sample"]


@pytest.mark.gpu
def test_headline_line_carries_the_auxiliary_legs():
    """The headline workload's line also carries the tiered workload's two
    tier parts and the packs under a concurrent producer."""
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print("case bench contract: qwen workload with auxiliary legs, 2 steps", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "2", "--warmup", "1",
                        "--no-cpu-baseline"], capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    d = json.loads([ln for ln in r.stdout.splitlines() if ln.strip()][-1])
    assert d["config"]["workload"] == "qwen-h3584"
    conc, tiers = d["aux"]["concurrent"], d["aux"]["tiered"]
    assert "error" not in conc and "error" not in tiers, d["aux"]
    assert conc["pack_alone_GBps"] > 0 and conc["pack_with_producer_GBps"] > 0 and conc["producer_writes"] > 0
    assert conc["producer_error"] is None
    assert tiers["config"]["workload"] == "tiered-h4096"
    assert 0 < tiers["hbm_tier"]["frac"] < 1 and tiers["hbm_tier"]["gather_ceiling_GBps"] > 0
    assert 0 < tiers["host_tier"]["GBps"] < tiers["host_tier"]["peak"] * 1.2
    assert 0 < tiers["host_tier_row_fraction"] < 1

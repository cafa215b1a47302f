"""The bench.py contract: one GPU only, counter-measured traffic read only from a summary
taken on the kernel's current sources, and (on a GPU) one JSON line with the fields the
driver reads."""
from __future__ import annotations

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_traffic_read_only_for_current_sources(tmp_path):
    prof = tmp_path / "p.md"
    h = bench.source_hash(bench.STEP_SOURCES)
    prof.write_text(f"source hash: `{h}`\n\nhbm bytes per launch: 123456\n")
    assert bench.measured_traffic(str(prof), bench.STEP_SOURCES) == {"bytes": 123456.0}
    stale = "0" * 16 if h != "0" * 16 else "1" * 16
    prof.write_text(f"source hash: `{stale}`\n\nhbm bytes per launch: 123456\n")
    assert bench.measured_traffic(str(prof), bench.STEP_SOURCES) is None
    assert bench.measured_traffic(str(tmp_path / "missing.md"), bench.STEP_SOURCES) is None


def test_committed_profiles_name_their_sources():
    for prof, files in ((bench.TRAFFIC_PROFILE, bench.SWEEP_SOURCES), (bench.STEP_PROFILE, bench.STEP_SOURCES),
                        (bench.VERIFY_PROFILE, bench.VERIFY_SOURCES), (bench.LOSS_PROFILE, bench.LOSS_SOURCES)):
        txt = open(prof).read()
        assert "source hash:" in txt and "hbm bytes per launch:" in txt, prof
        for f in files:
            assert os.path.exists(os.path.join(ROOT, "paper_2609_39972_amd", "csrc", f))


@pytest.mark.gpu
def test_bench_json_line():
    from gpu_util import say

    say("bench.py --steps 8 --warmup 2 --no-cpu-baseline --sweep-launches 8")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "8", "--warmup", "2",
                        "--no-cpu-baseline", "--sweep-launches", "8"], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "sweep_alone"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] >= 8 and d["value"] > 0 and d["unit"] == "trees/s"
    assert d["config"]["workload"] == "zipf-v151936-b32" and d["config"]["B"] == 32 and d["config"]["V"] == 151936
    rf = d["roofline"]
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert rf["kernel"] == bench.STEP_KERNEL
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    # trees/s = B / step time
    assert abs(d["value"] - 32 / (d["ms_per_step"] * 1e-3)) / d["value"] < 1e-3

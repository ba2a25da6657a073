"""bench.py's output contract.

CPU: more than one GPU is refused with a message and a non-zero status before anything
touches a device. GPU: one short run of a small round prints a single JSON line with the
fields the measurement relies on (metric, value, step time, roofline object of the
attention call, per-call times), and the value is the verified drafts over the step time.
"""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr or "single" in r.stderr
    assert r.stdout.strip() == ""


@pytest.mark.gpu
def test_short_run_prints_the_contract(monkeypatch, capsys):
    sys.path.insert(0, ROOT)
    import bench
    monkeypatch.setattr(sys, "argv", ["bench.py", "--workload", "c16_b16", "--steps", "3", "--warmup", "1",
                                      "--rotate", "1", "--cpu-seconds", "0", "--step-only"])
    bench.main()
    lines = [l for l in capsys.readouterr().out.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better", "scaling",
              "vs_baseline", "dtype", "data", "config", "roofline", "kernels", "cpu_baseline"):
        assert k in d, k
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1 and d["dtype"] == "bf16"
    assert d["value"] > 0 and d["ms_per_step"] > 0
    drafts = d["config"]["verified_drafts"]
    assert abs(d["value"] - drafts / (d["ms_per_step"] * 1e-3)) <= 1e-6 * d["value"]
    r = d["roofline"]
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == 8000.0
    assert abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-9 and 0.0 < r["frac"] < 1.0
    k = d["kernels"]
    assert k["attention_us"] > 0 and k["acceptance_us"] > 0
    assert (k["prepare_us"] or 0) > 0 or (k["budget_us"] or 0) > 0  # fused set-up, or budget and packing
    assert d["cpu_baseline"] is None  # --cpu-seconds 0

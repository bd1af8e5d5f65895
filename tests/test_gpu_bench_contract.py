"""bench.py's output contract on a small workload: one JSON line with the
metric, the whole-step throughput, the roofline object of the dominant kernel
(bound, achieved, peak, unit, frac = achieved / peak, traffic) and the CPU
baseline object (value, unit, cores, kind "oracle", sample)."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_json_line_contract():
    print("[case] bench.py --workload small", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--workload", "small", "--steps", "3",
                        "--warmup", "2", "--no-bandwidth", "--no-selection", "--no-cache", "--no-schedule",
                        "--no-frame-mask", "--no-shard", "--no-peaks", "--cpu-seconds", "2"],
                       capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 2 and d["higher_is_better"] is True
    assert d["config"]["workload"] == "small" and d["value"] > 0
    rl = d["roofline"]
    assert rl["bound"] == "mfma" and rl["unit"] == "TFLOP/s" and rl["peak"] == 2500.0
    assert rl["frac"] == pytest.approx(rl["achieved"] / rl["peak"], abs=1e-4)
    assert "traffic" in rl
    cb = d["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and cb["sample"]
    assert "speedup_vs_all_frame" in d and d["speedup_vs_all_frame"] > 1.0

"""The benchmark's one JSON line on a real run (the `small` workload, few
steps): the keys the contract names, the roofline object of the dominant
kernel class and the oracle baseline timed on the host, and the
arithmetic that ties them together."""
import json
import math
import os
import subprocess
import sys

import pytest

import cdsl_inputs as ci

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(600)
def test_bench_line_contract():
    cmd = [sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "small", "--steps", "2",
           "--warmup", "1", "--profile-steps", "1", "--phase-steps", "1", "--methods-steps", "0"]
    r = subprocess.run(cmd, cwd=ROOT, capture_output=True, text=True, timeout=540)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [ln for ln in r.stdout.splitlines() if ln.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    wl = ci.workload("small")
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1
    assert d["higher_is_better"] is True and d["vs_baseline"] is None
    assert d["config"]["workload"] == "small"
    # value = lookahead tokens verified per second = B k d / step time
    assert d["value"] == pytest.approx(wl.batch * wl.k * wl.d / (d["ms_per_step"] / 1e3), rel=2e-3)
    roof = d["roofline"]
    assert roof["bound"] in ("hbm", "mfma", "alu")
    assert roof["unit"] == ("TFLOP/s" if roof["bound"] == "mfma" else "GB/s")
    assert roof["peak"] == (2500.0 if roof["bound"] == "mfma" else 8000.0)
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], rel=1e-3, abs=1e-4)
    assert 0.0 < roof["frac"] < 1.0
    assert "traffic" in roof
    # the class's average launch, times its launches, fits inside the step
    assert roof["avg_launch_us"] * roof["launches"] / 1e3 <= d["ms_per_step"] * 1.5
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["unit"] == d["unit"]
    assert cpu["value"] > 0 and cpu["cores"] >= 1 and isinstance(cpu["sample"], str)
    assert math.isfinite(cpu["value"])

"""bench.py's one JSON line on a short run: the keys its readers rely on,
the roofline and cpu_baseline objects, and values that agree with each
other (value = query tokens / step time; frac = achieved / peak)."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("extra", [[], ["--config", "budget256", "--append", "separate"]], ids=["default", "mixed"])
def test_bench_line(extra):
    print(f"[gpu] bench.py --steps 3 {' '.join(extra)}", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "3", "--warmup", "1",
                        "--cpu-seconds", "0.5", *extra], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
              "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline", "measured_peaks"):
        assert k in line, k
    assert line["n_gpus"] == 1 and line["steps"] == 3 and line["higher_is_better"] is True
    assert line["value"] == pytest.approx(line["config"]["query_tokens"] / (line["ms_per_step"] * 1e-3), rel=1e-3)
    rf = line["roofline"]
    assert rf["bound"] in ("hbm", "mfma") and rf["unit"] in ("GB/s", "TFLOP/s")
    assert rf["frac"] == pytest.approx(rf["achieved"] / rf["peak"], rel=1e-3) and 0 < rf["frac"] < 1
    cb = line["cpu_baseline"]
    assert cb["kind"] == "oracle" and cb["value"] > 0 and cb["cores"] >= 1 and cb["sample"]
    assert "workload" in line["config"]
    if not extra:
        assert line["config"]["workload"].startswith("longctx") and rf["bound"] == "mfma"
    # the dominant half alone cannot take longer than the whole step
    assert rf["phase_ms"] <= line["ms_per_step"] * 1.02
    assert line["dtype"] == "bf16"

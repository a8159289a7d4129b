"""bench.py on the GPU prints one JSON line with the fields its benchmark
contract names, and figures that agree with each other: the throughput
with the time per pass, the roofline's achieved rate with its bytes and
launch time, its fraction with its peak, and a CPU-oracle baseline that
says what it timed.  Run on the small fp32 workload so it takes seconds."""
import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_line_contract():
    print("bench contract: tiny_fp32, 2 timed passes", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "tiny_fp32", "--steps",
                        "2", "--warmup", "1", "--cpu-seconds", "0.5", "--batched", "off"],
                       capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-3000:]
    lines = []
    for ln in r.stdout.splitlines():
        try:
            lines.append(json.loads(ln))
        except ValueError:
            continue
    assert len(lines) == 1, r.stdout[-3000:]
    d = lines[0]
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1
    assert d["higher_is_better"] is True and d["scaling"] in ("weak", "strong") and d["data"] == "synthetic"
    cfg = d["config"]
    assert cfg["workload"] == "tiny_fp32"
    # tokens/s = B * decode steps per pass / time per pass
    expect = cfg["B"] * cfg["decode_steps"] / (d["ms_per_step"] * 1e-3)
    assert abs(d["value"] - expect) <= 1e-3 * expect + 0.1
    rf = d["roofline"]
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in rf, key
    assert rf["bound"] == "hbm" and rf["unit"] == "GB/s" and rf["peak"] == 8000.0
    assert abs(rf["frac"] - rf["achieved"] / rf["peak"]) < 1e-3
    assert abs(rf["achieved"] - rf["bytes_per_launch"] / (rf["launch_us"] * 1e3)) <= 1e-2 * rf["achieved"]
    cb = d["cpu_baseline"]
    for key in ("value", "unit", "cores", "kind", "sample"):
        assert key in cb, key
    assert cb["kind"] == "oracle" and cb["unit"] == d["unit"] and cb["cores"] >= 1 and cb["value"] > 0

"""bench.py end to end on the GPU (small workload): one JSON line with the
fields the benchmark contract names, a roofline entry for the dominant
kernel and the oracle's CPU baseline.  Runs bench.py as a child process."""
import json
import os
import subprocess
import sys

import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_json_line():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print("[gpu-case] bench.py --workload trace512_tiny --steps 3 --warmup 1 --no-decode", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "bench.py"), "--workload", "trace512_tiny",
                        "--steps", "3", "--warmup", "1", "--no-decode"],
                       capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    lines = [x for x in r.stdout.splitlines() if x.startswith("{")]
    assert len(lines) == 1, r.stdout[-2000:]
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 3 and d["warmup"] == 1 and d["higher_is_better"] is True
    assert d["unit"] == "TFLOP/s" and d["dtype"] == "bf16" and d["data"] == "synthetic"
    assert d["config"]["workload"] == "trace512_tiny" and d["config"]["visible_pairs_per_head"] == 78080
    assert d["value"] > 0 and d["ms_per_step"] > 0
    assert d["value"] == pytest.approx(d["config"]["visible_tflop_per_step"] / (d["ms_per_step"] * 1e-3), rel=1e-9)
    roof = d["roofline"]
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s" and roof["peak"] == pytest.approx(2516.6)
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], rel=1e-9) and 0 < roof["frac"] < 1
    assert roof["kernel"] in ("fwd", "bwd_dkdv", "bwd_dq")
    cpu = d["cpu_baseline"]
    assert cpu["kind"] == "oracle" and cpu["unit"] == "TFLOP/s" and cpu["value"] > 0 and cpu["cores"] >= 1
    assert d["reprefill"]["time_ratio_reprefill_over_kv_streams"] > 0

"""Host-side logic of bench.py (no GPU): the visible-pair count behind the
FLOP rate, the source hash that gates the counter-derived traffic, the
counter scaling, and the one-GPU refusal."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

from oracle import attention as orc
from paper_2609_35750_amd import inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_visible_pairs_closed_form_matches_the_mask():
    """bench counts sum_j (min(e_j, L) - j) per trace; the oracle counts the explicit mask."""
    rng = np.random.default_rng(11)
    lengths = [0, 1, 77, 300, 0, 129]
    e = np.concatenate([inputs.evict_at_random(L, rng) for L in lengths if L])
    assert bench.visible_pairs(e, lengths) == orc.visible_pairs(e, lengths)
    wl = inputs.WORKLOADS["trace512_tiny"]
    assert bench.visible_pairs(wl.evict_at(), wl.lengths) == orc.visible_pairs(wl.evict_at(), wl.lengths) == 78080


def test_source_hash_ignores_comments_only():
    src = "int a; // note\n\n  b = a + 1;   \n// whole line\n"
    assert bench._code_only(src) == "int a;\n  b = a + 1;"
    assert bench._code_only(src.replace("note", "other note")) == bench._code_only(src)
    assert bench._code_only(src.replace("a + 1", "a + 2")) != bench._code_only(src)
    h = bench.kernel_source_hash()
    assert len(h) == 16 and h == bench.kernel_source_hash()


def test_traffic_summary_scales_by_the_copy(tmp_path, monkeypatch):
    """Counter KiB per dispatch, scaled so that the 1 GiB copy reads as 1 GiB each way."""
    def write(sub, rows):
        d = tmp_path / "out" / sub
        d.mkdir(parents=True)
        with open(d / "run_counter_collection.csv", "w") as fh:
            fh.write("Kernel_Name,Counter_Name,Counter_Value\n")
            for name, counter, kib in rows:
                fh.write(f"\"{name}\",{counter},{kib}\n")
    copy = "void at::native::copy_kernel(int)"
    write("cfetch", [(copy, "FETCH_SIZE", 2 * (1 << 20))] * 3)      # reads 2 GiB for 1 GiB moved: factor 1/2
    write("cwrite", [(copy, "WRITE_SIZE", 1 << 20)] * 3)
    fwd = "void kvs::fwd_kernel<128>(kvs::RowArgs)"
    write("fetch", [(fwd, "FETCH_SIZE", 1000.0), (fwd, "FETCH_SIZE", 3000.0)])
    write("write", [(fwd, "WRITE_SIZE", 500.0)])
    (tmp_path / "profiles").mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "0123456789abcdef")
    bench.traffic_summarize(str(tmp_path / "out"), "unit_test_workload")
    rec = json.load(open(tmp_path / "profiles" / "traffic_fwd_unit_test_workload.json"))
    assert rec["fetch_bytes_per_launch"] == pytest.approx(2000.0 * 1024 / 2)
    assert rec["write_bytes_per_launch"] == pytest.approx(500.0 * 1024)
    assert rec["bytes_per_launch"] == pytest.approx(2000.0 * 512 + 500.0 * 1024)
    assert rec["source_hash"] == "0123456789abcdef"
    assert sorted(os.listdir(tmp_path / "profiles")) == ["traffic_fwd_unit_test_workload.json"]


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2 and "one GPU" in r.stderr

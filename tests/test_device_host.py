"""Device helpers compiled for the host and run on the CPU (no GPU needed).

``tests/host/trace_clamp.hip`` checks the clamp the attention kernels apply to
trace offsets read from device memory (every addressed trace stays inside the
packed buffers and within max_seqlen; valid offsets pass unchanged) and the
tile-classifier switches of the ``*_ex`` calls.  ``tests/host/stager_bounds.hip``
checks the addressing of every staged tile: each LDS slot written once, every
source read inside the trace's rows, and rows inside the trace copied
unchanged through the swizzle."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or ("/opt/rocm/bin/hipcc" if os.path.exists("/opt/rocm/bin/hipcc") else None)


@pytest.mark.skipif(HIPCC is None, reason="hipcc not available")
def test_trace_clamp_and_class_switches(tmp_path):
    exe = str(tmp_path / "trace_clamp")
    cmd = [HIPCC, "-x", "hip", "--offload-host-only", "-O1", "-std=c++17", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2609_35750_amd", "csrc"), os.path.join(ROOT, "tests", "host", "trace_clamp.hip"),
           "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout + r.stderr


def _build_and_run(tmp_path, src, name):
    exe = str(tmp_path / name)
    cmd = [HIPCC, "-x", "hip", "--offload-host-only", "-O1", "-std=c++17", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2609_35750_amd", "csrc"), os.path.join(ROOT, "tests", "host", src), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return subprocess.run([exe], capture_output=True, text=True, timeout=120)


@pytest.mark.skipif(HIPCC is None, reason="hipcc not available")
def test_tile_copy_addressing(tmp_path):
    r = _build_and_run(tmp_path, "stager_bounds.hip", "stager_bounds")
    assert r.returncode == 0 and r.stdout.rstrip().endswith("ok"), r.stdout + r.stderr

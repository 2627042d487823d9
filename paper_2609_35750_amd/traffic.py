"""HBM traffic per kernel launch from rocprofv3 counter runs.

Two counter passes over the benchmark (``FETCH_SIZE``, then ``WRITE_SIZE``; KiB
per dispatch) and the same two passes over a plain device copy of known size
give the bytes each kernel moves to and from HBM, scaled by what the counters
read for the copy:

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT/fetch -o run -- python bench.py --no-cpu --no-reprefill --steps 2 --warmup 1
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT/write -o run -- python bench.py --no-cpu --no-reprefill --steps 2 --warmup 1
    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT/cfetch -o run -- python -m paper_2609_35750_amd.traffic copy
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT/cwrite -o run -- python -m paper_2609_35750_amd.traffic copy
    python -m paper_2609_35750_amd.traffic summarize OUT trace16k_gqa4 profiles

The summary step writes ``profiles/traffic_<kernel>_<workload>.json`` (read by
bench.py, together with a hash of the kernel source it was taken on) and
prints a markdown table.
"""
from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import sys
from collections import defaultdict

COPY_BYTES = 1 << 30
KERNELS = {"fwd_kernel": "fwd", "dkdv_kernel": "bwd_dkdv", "dq_kernel": "bwd_dq", "bwd_pre_kernel": "bwd_pre",
           "kstats_kernel": "classify", "paged_decode_kernel": "paged_decode"}


def _code_only(text: str) -> str:
    """Source without // comments, trailing blanks and empty lines: edits to
    comments do not change the kernels the counters were taken on."""
    out = []
    for line in text.splitlines():
        i = line.find("//")
        if i >= 0:
            line = line[:i]
        line = line.rstrip()
        if line:
            out.append(line)
    return "\n".join(out)


def kernel_source_hash(root: str) -> str:
    h = hashlib.sha256()
    for f in ("kvs_kernels.hip", "kvs_paged.hip", "kvs_device.h"):
        with open(os.path.join(root, "paper_2609_35750_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def copy_main() -> None:
    import torch

    src = torch.empty(COPY_BYTES // 2, dtype=torch.bfloat16, device="cuda:0").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES}))


def _per_kernel(d: str, counter: str):
    vals = defaultdict(list)
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            vals[r["Kernel_Name"]].append(float(r["Counter_Value"]) * 1024.0)   # KiB -> bytes
    return vals


def summarize(out: str, workload: str, profiles: str) -> None:
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    fetch, write = _per_kernel(os.path.join(out, "fetch"), "FETCH_SIZE"), _per_kernel(os.path.join(out, "write"), "WRITE_SIZE")
    cf, cw = _per_kernel(os.path.join(out, "cfetch"), "FETCH_SIZE"), _per_kernel(os.path.join(out, "cwrite"), "WRITE_SIZE")

    def biggest(vals):   # the copy kernel: the dispatch that moves the most bytes
        return max((sum(v) / len(v) for v in vals.values()), default=0.0)

    f_scale = COPY_BYTES / biggest(cf)
    w_scale = COPY_BYTES / biggest(cw)
    lines = [f"| kernel | FETCH_SIZE (MB/launch, scaled) | WRITE_SIZE (MB/launch, scaled) | launches |", "|---|---|---|---|"]
    src_hash = kernel_source_hash(root)
    for kname, vals in sorted(fetch.items()):
        short = next((v for k, v in KERNELS.items() if k in kname), None)
        if short is None:
            continue
        fb = sum(vals) / len(vals) * f_scale
        wv = write.get(kname, [0.0])
        wb = sum(wv) / len(wv) * w_scale
        lines.append(f"| `{kname.split('(')[0]}` | {fb / 1e6:.1f} | {wb / 1e6:.1f} | {len(vals)} |")
        rec = {"kernel": short, "workload": workload, "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
               "bytes_per_launch": fb + wb, "fetch_scale": f_scale, "write_scale": w_scale, "source_hash": src_hash}
        with open(os.path.join(profiles, f"traffic_{short}_{workload}.json"), "w") as fh:
            json.dump(rec, fh, indent=1)
    print(f"copy calibration: FETCH_SIZE x{f_scale:.4f}, WRITE_SIZE x{w_scale:.4f} (copy of {COPY_BYTES} bytes)")
    print("\n".join(lines))


if __name__ == "__main__":
    if len(sys.argv) >= 2 and sys.argv[1] == "copy":
        copy_main()
    elif len(sys.argv) >= 5 and sys.argv[1] == "summarize":
        summarize(sys.argv[2], sys.argv[3], sys.argv[4])
    else:
        print(__doc__)
        sys.exit(2)

"""Benchmark: eviction-masked attention forward + backward on one MI355X.

One step = the library's forward call plus its backward call over one
synthetic agent trace already resident in HBM (default: the 16,384-token
keep-all-summaries trace, Hq=32, Hkv=8, D=128).  Throughput counts visible
FLOPs only: 4*D per visible (query, key, q-head) triple in the forward and
10*D in the backward.

Prints one JSON line.  The value is timed over exactly K steps with nothing
else on the stream.  The same K steps are then run again with HIP events
around every kernel on its launch stream: for the kernel that takes the most
time, its algorithmic FLOPs per launch over its average launch duration
("roofline").  Also the fp64 CPU oracle timed on a bounded sample of the
same workload ("cpu_baseline").

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu]

HBM traffic per kernel launch (the ``traffic`` field of the roofline) comes
from two rocprofv3 counter passes over the benchmark (FETCH_SIZE, then
WRITE_SIZE; KiB per dispatch), each scaled by what the same counter reads for
a plain device copy of 1 GiB:

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT/fetch -o run -- python bench.py --no-cpu --no-reprefill --steps 2 --warmup 1
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT/write -o run -- python bench.py --no-cpu --no-reprefill --steps 2 --warmup 1
    rocprofv3 --pmc FETCH_SIZE --output-format csv -d OUT/cfetch -o run -- python bench.py --traffic-copy
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d OUT/cwrite -o run -- python bench.py --traffic-copy
    python bench.py --traffic-summarize OUT trace16k_gqa4

The summary step writes ``profiles/traffic_<kernel>_<workload>.json`` with a
hash of the kernel source it was taken on (a later kernel change voids it).
"""
import argparse
import csv
import dataclasses
import glob
import hashlib
import json
import math
import os
import sys
import time
from collections import defaultdict

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "eviction-masked attn fwd+bwd TFLOP/s (visible FLOPs) and % bf16 MFMA peak"
PEAK_BF16_TFLOPS = 2516.6          # MI355X dense bf16 MFMA, 256 CU x 2.4 GHz x 4096 FLOP/clk
# Algorithmic FLOPs per visible (query, key, q-head) triple, in units of D.
FLOPS_PER_VISIBLE = {"fwd": 4, "bwd_dkdv": 8, "bwd_dq": 2}   # dK/dV kernel: S, dP, dV, dK; dQ kernel: dQ
KERNELS = ("classify", "fwd", "bwd_pre", "bwd_dkdv", "bwd_dq")


def visible_pairs(evict_at, lengths):
    tot, off = 0, 0
    for L in lengths:
        e = np.minimum(evict_at[off:off + L].astype(np.int64), L)
        tot += int((e - np.arange(L)).sum())
        off += L
    return tot


# ---------------------------------------------------------------- HBM traffic from rocprofv3 counters
COPY_BYTES = 1 << 30
TRAFFIC_KERNELS = {"fwd_kernel": "fwd", "dkdv_kernel": "bwd_dkdv", "dq_kernel": "bwd_dq", "bwd_pre_kernel": "bwd_pre",
                   "kstats_kernel": "classify", "paged_decode_kernel": "paged_decode"}


def _code_only(text):
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


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("kvs_kernels.hip", "kvs_paged.hip", "kvs_device.h"):
        with open(os.path.join(ROOT, "paper_2609_35750_amd", "csrc", f), encoding="utf-8") as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def load_traffic(kernel, workload):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_launch")


def traffic_copy():
    """The calibration run: a plain device copy of COPY_BYTES, three times."""
    import torch

    src = torch.empty(COPY_BYTES // 2, dtype=torch.bfloat16, device="cuda:0").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES}))


def _counter_per_kernel(d, counter):
    vals = defaultdict(list)
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    vals[r["Kernel_Name"]].append(float(r["Counter_Value"]) * 1024.0)   # KiB -> bytes
    return vals


def traffic_summarize(out, workload):
    """Scaled FETCH/WRITE bytes per launch of each library kernel; writes
    profiles/traffic_<kernel>_<workload>.json and prints a markdown table."""
    fetch = _counter_per_kernel(os.path.join(out, "fetch"), "FETCH_SIZE")
    write = _counter_per_kernel(os.path.join(out, "write"), "WRITE_SIZE")
    cf = _counter_per_kernel(os.path.join(out, "cfetch"), "FETCH_SIZE")
    cw = _counter_per_kernel(os.path.join(out, "cwrite"), "WRITE_SIZE")
    biggest = lambda vals: max((sum(v) / len(v) for v in vals.values()), default=0.0)   # the copy dispatch
    f_scale, w_scale = COPY_BYTES / biggest(cf), COPY_BYTES / biggest(cw)
    lines = ["| kernel | FETCH_SIZE (MB/launch, scaled) | WRITE_SIZE (MB/launch, scaled) | launches |", "|---|---|---|---|"]
    src_hash = kernel_source_hash()
    for kname, vals in sorted(fetch.items()):
        short = next((v for k, v in TRAFFIC_KERNELS.items() if k in kname), None)
        if short is None:
            continue
        fb = sum(vals) / len(vals) * f_scale
        wv = write.get(kname, [0.0])
        wb = sum(wv) / len(wv) * w_scale
        lines.append(f"| `{kname.split('(')[0]}` | {fb / 1e6:.1f} | {wb / 1e6:.1f} | {len(vals)} |")
        rec = {"kernel": short, "workload": workload, "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
               "bytes_per_launch": fb + wb, "fetch_scale": f_scale, "write_scale": w_scale, "source_hash": src_hash}
        with open(os.path.join(ROOT, "profiles", f"traffic_{short}_{workload}.json"), "w") as fh:
            json.dump(rec, fh, indent=1)
    print(f"copy calibration: FETCH_SIZE x{f_scale:.4f}, WRITE_SIZE x{w_scale:.4f} (copy of {COPY_BYTES} bytes)")
    print("\n".join(lines))


def measured_mfma_rate():
    """Dense bf16 matrix-core rate the device sustains on changing operands
    (TFLOP/s), from the benchmark-only probe library built next to libkvs."""
    import ctypes

    import torch

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2609_35750_amd", "libkvs_bench.so"))
    lib.kvs_bench_mfma_rate.restype = ctypes.c_int
    lib.kvs_bench_mfma_rate.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.c_void_p]
    out = ctypes.c_double(0.0)
    rc = lib.kvs_bench_mfma_rate(ctypes.byref(out), torch.cuda.current_stream().cuda_stream)
    if rc != 0:
        raise RuntimeError(f"matrix-core probe failed ({rc})")
    return float(out.value)


# The paper's own end-to-end numbers, for context only (Abstract; Section 1;
# Section 5.2; the hardware of Section 4 and the training-details table).
PAPER_CONTEXT = {
    "kind": "context, not a target: end-to-end RL training wall-clock (generation + trainer forward/backward) "
            "of KV-streams over re-prefill compaction, on the paper's hardware; reprefill.time_ratio below is "
            "the attention-kernel analogue on one MI355X",
    "claims": [
        {"speedup": "2.6x to 5x training wall-clock, three compaction strategies", "where": "Abstract"},
        {"speedup": "5x on TextWorld, 1.3x on ALFWorld", "where": "Section 1"},
        {"speedup": "3x to peak (Sliding Window, KV-streams vs full context) on SWE", "where": "Section 5.2"},
    ],
    "hardware": {"TextWorld": "one 8-GPU H100 node (4 inference, 4 trainer)",
                 "ALFWorld": "4 A100 GPUs (1 inference, 3 trainer)",
                 "SWE": "one 8-GPU GB200 node (4 inference, 4 trainer)"},
}


def reprefill_batch(wl):
    """The varlen batch re-prefill compaction would run for the same rollouts:
    per trace, the fresh causal traces of inputs.reprefill_traces."""
    from paper_2609_35750_amd import inputs

    lengths, extra_exact, extra_formula = [], 0, 0.0
    e_all, off = wl.evict_at(), 0
    for L in wl.lengths:
        tr = inputs.reprefill_traces_from_evict(e_all[off:off + L])
        off += L
        lengths += [len(t) for t in tr]
        extra_exact += sum(len(t) for t in tr) - L
        # N r / (B - r) (Section 2): N generated entries, r kept and B - r new entries per compaction (means)
        if len(tr) > 1:
            # r: entries kept at each compaction; B - r: entries generated between two compactions
            # (new parts of the traces that end in a compaction; trace 0 minus the prompt if there is one)
            news, kept = [], []
            pos = len(tr[0])
            for t in tr[1:]:
                k = int(np.sum(t < pos))
                kept.append(k)
                news.append(len(t) - k)
                pos += len(t) - k
            gaps = news[:-1] if len(news) > 1 else [len(tr[0]) - min(wl.p, L)]
            extra_formula += (L - wl.p) * float(np.mean(kept)) / float(np.mean(gaps))
    return lengths, extra_exact, extra_formula


def time_steps(step, warmup, steps):
    import torch

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / steps


def reprefill_compare(wl, kvs, warmup, steps, kvs_ms):
    """Kernel-level analogue of the paper's re-prefill comparison (Section 2,
    "Prefill-compaction"): the same library, forward + backward, over the
    causal traces re-prefill compaction would run instead of one masked trace."""
    import torch

    from paper_2609_35750_amd import inputs

    lengths, extra_exact, extra_formula = reprefill_batch(wl)
    n = int(sum(lengths))
    dev = torch.device("cuda:0")
    qs = 1.0 / math.sqrt(wl.D) if wl.q_prescaled else 1.0
    q = inputs.randn_bf16((n, wl.Hq, wl.D), wl.seed * 16 + 9, qs).to(dev)
    k = inputs.randn_bf16((n, wl.Hkv, wl.D), wl.seed * 16 + 10).to(dev)
    v = inputs.randn_bf16((n, wl.Hkv, wl.D), wl.seed * 16 + 11).to(dev)
    do = inputs.randn_bf16((n, wl.Hq, wl.D), wl.seed * 16 + 12).to(dev)
    ev = torch.from_numpy(np.concatenate([np.full(L, L, dtype=np.int32) for L in lengths])).to(dev)   # never evicted
    cu_np = np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)
    cu = torch.from_numpy(cu_np).to(dev)
    T = int(max(lengths))
    kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale, cu, T)   # validates cu_seqlens once
    o = torch.empty_like(q)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    lse = None

    def step():
        nonlocal lse
        _, lse = kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale, cu, T, out=o, lse=lse, check_cu=False)
        kvs.kvs_evict_attn_bwd(do, q, k, v, o, lse, ev, wl.softmax_scale, cu, T, dq=dq, dk=dk, dv=dv, check_cu=False)

    ms = time_steps(step, warmup, steps)
    pairs = int(sum(L * (L + 1) // 2 for L in lengths))
    return {"traces": len(lengths), "tokens": n, "tokens_kv_streams": wl.ntok,
            "extra_tokens_exact": int(extra_exact), "extra_tokens_formula_Nr_over_B_minus_r": round(extra_formula, 1),
            "visible_pairs_per_head": pairs, "ms_per_step": ms, "kv_streams_ms_per_step": kvs_ms,
            "time_ratio_reprefill_over_kv_streams": ms / kvs_ms}


PEAK_HBM_GBS = 8000.0   # MI355X HBM3E


def paged_decode_bench(warmup, steps, S=64, block_size=16):
    """Decode over the streamed paged KV cache (the inference side): S rollouts
    shaped like the 16k keep-all trace (Hq=32, Hkv=8, D=128, 16-token blocks)
    are streamed through one cache segment by segment (turns and summary
    appended, then the turns evicted, freed blocks reused across rollouts),
    and one query per rollout is decoded at the last token.  HBM-bound: the
    algorithmic bytes are the live K and V entries read once (plus Q and O)."""
    import torch

    from paper_2609_35750_amd import inputs, paged
    from paper_2609_35750_amd import kvs

    L, p, w, s_, Hq, Hkv, D = 16384, 1024, 4096, 512, 32, 8, 128
    e = inputs.evict_at_layout(L, p, w, s_, "keep_all")
    dev = torch.device("cuda:0")
    max_blocks = (L + block_size - 1) // block_size + 1
    live_max = int(np.sum(np.minimum(e, L) > L - 1))
    nb = S * ((live_max + w + s_) // block_size + 4)
    cache = paged.PagedKVCache(nb, block_size, S, max_blocks, Hkv, D, device=dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(1234)
    # eviction events: positions evicted at each time
    ev_t = {}
    for j, x in enumerate(np.minimum(e, L)):
        if x < L:
            ev_t.setdefault(int(x), []).append(j)
    cuts = sorted(set(ev_t) | {L})
    for sq in range(S):
        t0 = 0
        for t1 in cuts:
            if t0 < t1:
                n = t1 - t0
                kn = torch.randn((n, Hkv, D), generator=gen, device=dev).to(torch.bfloat16)
                vn = torch.randn((n, Hkv, D), generator=gen, device=dev).to(torch.bfloat16)
                cache.append(sq, np.arange(t0, t1), kn, vn)
            if t1 < L:
                cache.evict(sq, ev_t[t1])
            t0 = t1
    live = sum(cache.bm.live(sq) for sq in range(S))
    q = torch.randn((S, Hq, D), generator=gen, device=dev).to(torch.bfloat16)
    o = torch.empty_like(q)
    lse = torch.empty((S, Hq), dtype=torch.float32, device=dev)
    for _ in range(warmup):
        cache.decode(q, 1.0 / math.sqrt(D), out=o, lse=lse)
    torch.cuda.synchronize()
    kvs.kvs_prof_reset()
    kvs.kvs_prof_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        cache.decode(q, 1.0 / math.sqrt(D), out=o, lse=lse)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    kvs.kvs_prof_enable(False)
    n, ms = kvs.kvs_prof_read("paged_decode")
    kvs.kvs_prof_reset()
    kern_ms = ms / max(n, 1)
    kv_bytes = live * Hkv * D * 2 * 2
    io_bytes = 2 * S * Hq * D * 2 + S * Hq * 4
    algo = kv_bytes + io_bytes
    achieved = algo / (kern_ms * 1e-3) / 1e9
    return {
        "workload": f"{S} rollouts of the 16k keep-all trace (Hq={Hq}, Hkv={Hkv}, D={D}) decoded at token {L - 1}",
        "block_size": block_size, "live_entries": live, "cache_blocks": nb,
        "call_ms": (t1 - t0) * 1e3 / steps, "kernel_ms": kern_ms,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": load_traffic("paged_decode", "trace16k_gqa4"),
                     "kernel": "paged_decode", "algorithmic_bytes_per_launch": algo},
    }


def cp_shard_bench(wl, tensors, evict_at, n_shards, warmup, steps, full_ms):
    """The single-GPU part of context parallelism: the trace's query rows cut
    into n_shards ranges of about equal work at segment starts, each shard's forward + backward run
    on its local trace (gathered live keys, then its own tokens) with inputs
    resident, timed one shard after another.  Reports the slowest shard (the
    compute time of an n-GPU step, before communication) and the keys the
    forward's all-gather and the backward's reduce-scatter would move."""
    import torch

    from paper_2609_35750_amd import inputs, kvs, shard

    dev = torch.device("cuda:0")
    plans = shard.plan_trace(evict_at, n_shards, inputs.segment_starts(wl.T, wl.p, wl.w, wl.s), balance=True)
    q, k, v, do = (tensors[x].to(dev) for x in ("q", "k", "v", "do"))
    times = []
    for p in plans:
        idx = torch.from_numpy(p.keys).to(dev)
        zq = torch.zeros((p.n_g, wl.Hq, wl.D), dtype=q.dtype, device=dev)
        shp = lambda x: x.contiguous().view(1, p.length, x.shape[1], wl.D)
        ql, dol = shp(torch.cat([zq, q[p.r0:p.r1]])), shp(torch.cat([zq, do[p.r0:p.r1]]))
        kl, vl = shp(k.index_select(0, idx)), shp(v.index_select(0, idx))
        ev = torch.from_numpy(p.evict_local).to(dev).view(1, p.length)
        o = torch.empty_like(ql)
        dq, dk, dv = torch.empty_like(ql), torch.empty_like(kl), torch.empty_like(vl)
        lse = None

        def step():
            nonlocal lse
            _, lse = kvs.kvs_evict_attn_fwd(ql, kl, vl, ev, wl.softmax_scale, out=o, lse=lse)
            kvs.kvs_evict_attn_bwd(dol, ql, kl, vl, o, lse, ev, wl.softmax_scale, dq=dq, dk=dk, dv=dv)

        times.append(time_steps(step, warmup, steps))
    vol = shard.exchange_volume(plans, wl.Hkv, wl.D)
    return {"shards": len(plans), "rows": [p.r1 - p.r0 for p in plans], "gathered_keys": [p.n_g for p in plans],
            "ms_per_shard": [round(t, 4) for t in times], "max_shard_ms": max(times), "full_trace_ms": full_ms,
            "compute_speedup_vs_one_gpu": full_ms / max(times), "all_gather_bytes_kv": vol["bytes_kv"]}


def cpu_baseline(wl, tensors, evict_at, min_seconds=10.0):
    """The fp64 oracle as it stands, timed one q-head at a time (with its KV
    head) over the whole workload until at least `min_seconds` have passed."""
    from oracle import attention as orc

    cu = wl.cu_seqlens() if wl.varlen else None
    per_head = visible_pairs(evict_at, wl.lengths)
    heads, dt = 0, 0.0
    while heads < wl.Hq and dt < min_seconds:
        h = heads
        g = h // wl.G
        sl = slice(h, h + 1)
        t0 = time.perf_counter()
        orc.backward(tensors["q"][:, sl], tensors["k"][:, g:g + 1], tensors["v"][:, g:g + 1], evict_at,
                     wl.softmax_scale, tensors["do"][:, sl], cu_seqlens=cu)
        dt += time.perf_counter() - t0
        heads += 1
    flops = 14 * wl.D * heads * per_head
    try:
        from threadpoolctl import threadpool_info

        cores = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        cores = len(os.sched_getaffinity(0))
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"fp64 forward+backward of q-heads 0..{heads - 1} (each with its KV head) over the whole "
                      f"{wl.name} workload ({flops / 1e12:.3f} visible TFLOP in {dt:.1f} s)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="trace16k_gqa4")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle timing")
    ap.add_argument("--no-reprefill", action="store_true", help="skip the re-prefill comparison")
    ap.add_argument("--no-decode", action="store_true", help="skip the paged-cache decode measurement")
    ap.add_argument("--cp-shards", type=int, default=0,
                    help="also time the trace cut into this many context-parallel shards (one after another)")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of one step captured as a HIP graph (no host launch gaps)")
    ap.add_argument("--hq", type=int, default=0,
                    help="diagnostics: override the workload's q-head count (a multiple of its KV heads)")
    ap.add_argument("--d", type=int, default=0, choices=(0, 64, 128),
                    help="diagnostics: override the workload's head dimension (64 or 128)")
    ap.add_argument("--traffic-copy", action="store_true", help="run the 1 GiB copy that calibrates the counters")
    ap.add_argument("--traffic-summarize", nargs=2, metavar=("OUT", "WORKLOAD"),
                    help="summarise FETCH/WRITE counter runs under OUT into profiles/")
    args = ap.parse_args()
    if args.traffic_summarize:
        traffic_summarize(*args.traffic_summarize)
        return
    if args.traffic_copy:
        traffic_copy()
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (--cp-shards N times the "
              "context-parallel shards of the trace one after another on one GPU); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_35750_amd import inputs, kvs

    wl = inputs.WORKLOADS[args.workload]
    if args.hq:
        if args.hq % wl.Hkv:
            sys.exit(f"--hq must be a multiple of the workload's {wl.Hkv} KV heads")
        wl = dataclasses.replace(wl, Hq=args.hq, name=f"{wl.name}_hq{args.hq}")
    if args.d and args.d != wl.D:
        wl = dataclasses.replace(wl, D=args.d, name=f"{wl.name}_d{args.d}")
    dev = torch.device("cuda:0")
    tensors = inputs.make_tensors(wl)
    e = wl.evict_at()
    vis = visible_pairs(e, wl.lengths)
    f_fwd = 4 * wl.D * wl.Hq * vis
    f_bwd = 10 * wl.D * wl.Hq * vis

    if wl.varlen:
        q, k, v, do = (tensors[x].to(dev) for x in ("q", "k", "v", "do"))
        ev = torch.from_numpy(e).to(dev)
        cu = torch.from_numpy(wl.cu_seqlens()).to(dev)
        kw = dict(cu_seqlens=cu, max_seqlen=wl.T, check_cu=False)
        kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale, cu, wl.T)  # validates cu_seqlens once
    else:
        shp = lambda x: x.to(dev).view(1, wl.T, x.shape[1], wl.D)
        q, k, v, do = (shp(tensors[x]) for x in ("q", "k", "v", "do"))
        ev = torch.from_numpy(e).to(dev).view(1, wl.T)
        kw = {}

    o = torch.empty_like(q)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    lse = None

    def step():
        nonlocal lse
        _, lse = kvs.kvs_evict_attn_fwd(q, k, v, ev, wl.softmax_scale, out=o, lse=lse, **kw)
        kvs.kvs_evict_attn_bwd(do, q, k, v, o, lse, ev, wl.softmax_scale, dq=dq, dk=dk, dv=dv, **kw)

    for _ in range(args.warmup):
        step()
    timed = step
    if args.graph:
        # One step (forward call + backward call) captured as a HIP graph and
        # replayed: the same kernels with the same arguments, without the host
        # launch gaps between them.
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        for _ in range(args.warmup):
            graph.replay()
        timed = graph.replay
    # Timed region: exactly K steps, nothing else on the stream.
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        timed()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    # The same K steps again, each bracketed by HIP events on the stream the
    # library launches on: the median per-step time of the calls.
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for ea, eb in evs:
        ea.record()
        timed()
        eb.record()
    torch.cuda.synchronize()
    ms_median_events = float(np.median([ea.elapsed_time(eb) for ea, eb in evs]))
    # The same K steps again with HIP events around every kernel on its launch
    # stream (per-kernel durations for the roofline).  The events sit between
    # the kernels and cost launch gaps, so they stay out of the timed region.
    kvs.kvs_prof_reset()
    kvs.kvs_prof_enable(True)
    torch.cuda.synchronize()
    tp0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    tp1 = time.perf_counter()
    kvs.kvs_prof_enable(False)
    per_kernel = {}
    for name in KERNELS:
        n, ms = kvs.kvs_prof_read(name)
        if n:
            per_kernel[name] = {"launches": n, "avg_ms": ms / n}
    kvs.kvs_prof_reset()

    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = (f_fwd + f_bwd) / (ms_per_step * 1e-3) / 1e12

    dom = max((k_ for k_ in per_kernel if k_ in FLOPS_PER_VISIBLE), key=lambda k_: per_kernel[k_]["avg_ms"])
    flops_launch = FLOPS_PER_VISIBLE[dom] * wl.D * wl.Hq * vis
    achieved = flops_launch / (per_kernel[dom]["avg_ms"] * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_BF16_TFLOPS, "traffic": load_traffic(dom, wl.name),
                "kernel": dom, "avg_ms": per_kernel[dom]["avg_ms"],
                "algorithmic_flops_per_launch": flops_launch}

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "launch": "hip_graph" if args.graph else "eager",
        "config": {"workload": wl.name, "traces": wl.B, "tokens": wl.ntok, "Hq": wl.Hq, "Hkv": wl.Hkv, "D": wl.D,
                   "layout": {"prompt": wl.p, "turns": wl.w, "summary": wl.s, "strategy": wl.strategy},
                   "visible_pairs_per_head": vis, "visible_tflop_per_step": (f_fwd + f_bwd) / 1e12},
        "pct_of_bf16_peak": 100.0 * value / PEAK_BF16_TFLOPS,
        "kernels_ms": {k_: round(v_["avg_ms"], 4) for k_, v_ in per_kernel.items()},
        "ms_per_step_with_kernel_events": (tp1 - tp0) * 1e3 / args.steps,
        "ms_per_step_median_hip_events": ms_median_events,
        "roofline": roofline,
    }
    out["value_strict_12D"] = 12 * wl.D * wl.Hq * vis / (ms_per_step * 1e-3) / 1e12   # no recompute counted
    measured_peak = measured_mfma_rate()
    out["measured_mfma_peak_tflops"] = measured_peak
    out["pct_of_measured_peak"] = 100.0 * value / measured_peak
    roofline["frac_of_measured_peak"] = achieved / measured_peak
    if not args.no_reprefill:
        out["reprefill"] = reprefill_compare(wl, kvs, args.warmup, args.steps, ms_per_step)
    out["paper_context"] = PAPER_CONTEXT
    if args.cp_shards > 0 and not wl.varlen:
        out["cp_shards"] = cp_shard_bench(wl, tensors, e, args.cp_shards, args.warmup, args.steps, ms_per_step)
    if not args.no_decode:
        out["paged_decode"] = paged_decode_bench(args.warmup, args.steps)
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(wl, tensors, e)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

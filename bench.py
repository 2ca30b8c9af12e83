"""Benchmark: decode steps of one HySparse2 hybrid block on one MI355X.

A step is the whole hot path over one batch of resident synthetic inputs:
one full-attention layer with pooled scores and forced-window + top-k
selection (hs2_full_attn_score_select), then the block's sparse layers
(hs2_sparse_attn), each with its own queries, reusing the cache and indices.

Default workload: 8-query verify chunk per sequence, batch 4, 131072-token
context, 32 query / 4 KV heads, head_dim 128, top-k 4096 + window 256,
1 full + 3 sparse layers (bf16 cache, fp32 accumulation).

Prints one JSON line (rank 0, N = 1).  Extra fields: achieved algorithmic
GB/s of the step, the roofline of the dominant kernel (full-attention split
kernel) from HIP events around its launches, per-kernel averages, and the
CPU oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "hybrid-block decode tokens/sec and achieved HBM GB/s at 128K ctx, 1 MI355X"
HBM_PEAK_GBS = 8000.0
DEFAULT_WORKLOAD = "chunk8_128k_b4"
KERNEL_SOURCES = ["paper_2609_26368_amd/csrc/hs2_kernels.hip", "paper_2609_26368_amd/csrc/hs2_device.h",
                  "paper_2609_26368_amd/csrc/hs2_api.hip"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fa_split_traffic_{workload}.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the code of the kernel sources (comments and blank space do not
    count: they do not change what runs)."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p)) as f:
            src = f.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="budget of the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sa-sink-gate", action="store_true",
                    help="sparse layers with per-head sink logits and sigmoid output gates (hs2_sparse_attn_ex)")
    ap.add_argument("--kv", choices=("bf16", "fp8"), default="bf16",
                    help="cache format: bf16, or OCP E4M3 bytes with one scale per KV head (the _fp8 entry points)")
    ap.add_argument("--block", type=int, default=0,
                    help="block-level selection with blocks of this many tokens (hs2_full_attn_score_select_blocks)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step in a HIP graph and time its replays (no per-kernel host launches)")
    ap.add_argument("--cold", action="store_true",
                    help="evict the caches (read a 1 GiB buffer) before every step; steps timed one by one")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain device copy of COPY_BYTES (counter calibration)")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                    help="turn rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE runs into the traffic record of fa_split")
    return ap.parse_args()


COPY_BYTES = 1 << 30


def copy_calibration():
    """A plain copy of COPY_BYTES, 5 times: its FETCH_SIZE / WRITE_SIZE per dispatch
    give the factor from counter units to bytes."""
    import torch
    src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": COPY_BYTES, "launches": 5}))


def _pmc_per_kernel(d, counter):
    import csv
    import glob
    import re
    vals = {}
    for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        per = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            key = (r["Dispatch_Id"], re.sub(r"\(.*", "", r["Kernel_Name"]))
            per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
        for (_, name), v in per.items():
            vals.setdefault(name, []).append(v)
    return {k: sum(v) / len(v) for k, v in vals.items()}


def summarize_pmc(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, workload):
    fetch = _pmc_per_kernel(fetch_dir, "FETCH_SIZE")
    write = _pmc_per_kernel(write_dir, "WRITE_SIZE")
    cf = _pmc_per_kernel(copy_fetch_dir, "FETCH_SIZE")
    cw = _pmc_per_kernel(copy_write_dir, "WRITE_SIZE")
    copy_name = max(cf, key=lambda k: cf[k])  # the copy kernel dominates its run
    f_fac = COPY_BYTES / (cf[copy_name] * 1024.0)
    w_fac = COPY_BYTES / (cw[copy_name] * 1024.0)
    fa = [k for k in fetch if "k_fa_" in k]
    rec = {"workload": workload, "source_hash": kernel_source_hash(), "kernel": fa[0] if fa else None,
           "copy_kernel": copy_name, "fetch_factor": f_fac, "write_factor": w_fac,
           "fetch_bytes_per_launch": fetch[fa[0]] * 1024 * f_fac if fa else None,
           "write_bytes_per_launch": write[fa[0]] * 1024 * w_fac if fa else None}
    rec["bytes_per_launch"] = (rec["fetch_bytes_per_launch"] or 0) + (rec["write_bytes_per_launch"] or 0)
    rec["per_kernel_bytes"] = {k: {"fetch": fetch.get(k, 0) * 1024 * f_fac, "write": write.get(k, 0) * 1024 * w_fac}
                               for k in sorted(set(fetch) | set(write))}
    out = TRAFFIC_FILE.format(workload=workload)
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps(rec))


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.workload + ("_fp8" if args.kv == "fp8" else ""))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (run with --gpus 1)",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_26368_amd import hs2
    from paper_2609_26368_amd import workloads as W

    if not os.path.exists(hs2.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    w = W.WORKLOADS[args.workload]
    t = time.perf_counter()
    inp = W.make_inputs(w, kv=args.kv)
    log(f"[bench] inputs {w.name} ({args.kv} cache) generated in {time.perf_counter() - t:.1f}s lens={inp.lens.tolist()}")
    B, C, Hq, Hkv, D = w.batch, w.n_queries, w.n_q_heads, w.n_kv_heads, w.head_dim
    Lmax = inp.K.shape[2]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    if args.kv == "fp8":
        K, V = torch.from_numpy(inp.K).to(dev), torch.from_numpy(inp.V).to(dev)
        kv_scales = (torch.from_numpy(inp.k_scale).to(dev), torch.from_numpy(inp.v_scale).to(dev))
    else:
        K, V = to_dev(inp.K), to_dev(inp.V)
        kv_scales = None
    q_fa = to_dev(inp.q_fa)
    q_sa = [to_dev(x) for x in inp.q_sa]
    lens = torch.from_numpy(inp.lens).to(dev)
    blk = hs2.HybridBlock(B, C, Hq, Hkv, D, Lmax, w.k, w.window, device=dev)
    out = torch.empty((B, C, Hq, D), dtype=torch.bfloat16, device=dev)
    idx = torch.empty((B, Hkv, C, w.slots), dtype=torch.int32, device=dev)
    sa_out = [torch.empty_like(out) for _ in q_sa]
    stream = torch.cuda.current_stream()
    sinks, gates = [None] * len(q_sa), [None] * len(q_sa)
    if args.sa_sink_gate:  # synthetic per-layer sink logits and gate logits
        g = torch.Generator(device="cpu").manual_seed(2609)
        sinks = [torch.randn(Hq, generator=g).to(dev) for _ in q_sa]
        gates = [torch.randn((B, C, Hq, D), generator=g).to(torch.bfloat16).to(dev) for _ in q_sa]

    def step_on(st):
        blk.full(q_fa, K, V, lens, out=out, idx=idx, stream=st, kv_scales=kv_scales, block=args.block)
        for qs, o, sk, gt in zip(q_sa, sa_out, sinks, gates):
            blk.sparse(qs, K, V, lens, idx, out=o, stream=st, sink=sk, gate=gt, kv_scales=kv_scales)

    def step():
        step_on(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} steps done")
    run_step = step
    if args.graph:  # one step captured after the warmup (the library's set-up is done by then)
        graph, cap = torch.cuda.CUDAGraph(), torch.cuda.Stream()
        cap.wait_stream(stream)
        with torch.cuda.graph(graph, stream=cap):
            step_on(cap)
        torch.cuda.synchronize()
        run_step = graph.replay
    tokens = B * C
    # evicting by reading 1 GiB (a write would leave dirty lines whose
    # write-back then overlaps the timed step)
    flush = torch.ones(1 << 28, dtype=torch.int32, device=dev) if args.cold else None
    if not args.cold:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record(stream)
        for _ in range(args.steps):
            run_step()
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ev_ms = e0.elapsed_time(e1)
        ms_per_step = ev_ms / args.steps
        value = tokens * args.steps / wall
        log(f"[bench] timed {args.steps} steps: wall {wall * 1e3:.2f} ms, events {ev_ms:.2f} ms")

    # one event pair per step: percentiles (and, cold, the timing itself: the
    # cache-evicting write before each step stays outside its events)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    for a_, b_ in ev:
        if flush is not None:
            flush.amax()
        a_.record(stream)
        run_step()
        b_.record(stream)
    torch.cuda.synchronize()
    per_step = np.array([a_.elapsed_time(b_) for a_, b_ in ev])
    if args.cold:
        ms_per_step = float(per_step.mean())
        value = tokens / (ms_per_step * 1e-3)
        log(f"[bench] timed {args.steps} cold steps: {ms_per_step:.4f} ms mean")
    pct = {f"p{q}": round(float(np.percentile(per_step, q)), 4) for q in (10, 50, 90)}

    # per-kernel durations (HIP events recorded by the library around each launch, same stream)
    hs2.hs2_timing_enable(True)
    hs2.hs2_timing_reset()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    per = hs2.hs2_timing_read()
    hs2.hs2_timing_enable(False)
    kernels = {name: {"launches": n, "avg_us": 1e3 * ms / n} for name, (n, ms) in per.items()}

    # algorithmic bytes (what the method must move; scratch and partials excluded)
    L = inp.lens.astype(np.int64)
    kv_row = 2 * D * (1 if args.kv == "fp8" else 2)  # K and V row of one token and KV head
    q_bytes = B * C * Hq * D * 2
    fa_bytes = int(L.sum()) * Hkv * kv_row + q_bytes
    idx_h = idx.cpu().numpy()
    uniq = sum(np.unique(idx_h[b, g][idx_h[b, g] >= 0]).size for b in range(B) for g in range(Hkv))
    step_bytes = (fa_bytes + q_bytes + idx_h.nbytes) + w.n_sparse * (uniq * kv_row + 2 * q_bytes + idx_h.nbytes)
    fa_avg_s = kernels["fa_split"]["avg_us"] * 1e-6
    achieved = fa_bytes / fa_avg_s / 1e9
    traffic = None  # HBM bytes per launch from calibrated counters, if taken on these kernels
    tf = TRAFFIC_FILE.format(workload=w.name + ("_fp8" if args.kv == "fp8" else ""))
    if os.path.exists(tf):
        with open(tf) as f:
            trec = json.load(f)
        if trec.get("source_hash") == kernel_source_hash():
            traffic = int(trec["bytes_per_launch"])
    roofline = {"kernel": "fa_split", "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "algorithmic_bytes_per_launch": fa_bytes}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, inp, args.cpu_seconds)

    rec = {"metric": METRIC, "value": round(value, 2), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": w.name, "batch": B, "ctx": w.ctx, "ctx_min": w.ctx_min or w.ctx,
                      "queries_per_seq": C, "q_heads": Hq, "kv_heads": Hkv, "head_dim": D, "k": w.k,
                      "window": w.window, "sparse_layers": w.n_sparse, "needles": w.needles,
                      "kv_cache": "e4m3" if args.kv == "fp8" else "bf16",
                      "selection": f"block{args.block}" if args.block else "token",
                      "launch": "graph" if args.graph else "eager",
                      "caches": "evicted before every step" if args.cold else "as left by the previous step",
                      **({"sa_sink_gate": True} if args.sa_sink_gate else {})},
           "achieved_gbps": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
           "algorithmic_bytes_per_step": int(step_bytes),
           "roofline": roofline,
           "step_ms_percentiles": pct,
           "kernels_avg_us": {k: round(v["avg_us"], 2) for k, v in kernels.items()},
           "cpu_baseline": cpu}
    print(json.dumps(rec), flush=True)


def cpu_baseline(w, inp, budget_s: float) -> dict:
    """The oracle on (sequence, KV head) groups of the same inputs until the
    budget is spent; scaled to tokens/s of whole steps."""
    from oracle import hs2_oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        threads = 1
    groups_all = [(b, g) for b in range(w.batch) for g in range(w.n_kv_heads)]
    n, t0 = 0, time.perf_counter()
    while True:  # cycle over the groups (again if a step's groups take less than the budget)
        O.hybrid_block(inp.q_fa, inp.q_sa, inp.K, inp.V, inp.lens, w.k, w.window,
                       groups=[groups_all[n % len(groups_all)]], k_scale=inp.k_scale, v_scale=inp.v_scale)
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    step_s = el * len(groups_all) / n
    log(f"[bench] oracle: {n} group evaluations ({len(groups_all)} per step) in {el:.1f}s")
    return {"value": round(w.batch * w.n_queries / step_s, 4), "unit": "tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{n} (sequence, KV head) group evaluations, cycling over the {len(groups_all)} groups of "
                      f"one step, full context, {el:.1f}s; scaled by {len(groups_all)}/{n}"}


if __name__ == "__main__":
    main()

"""Benchmark: decode steps of one HySparse2 hybrid block on one MI355X.

A step is the whole hot path over one batch of resident synthetic inputs:
one full-attention layer with pooled scores and forced-window + top-k
selection (hs2_full_attn_score_select), then the block's sparse layers
(hs2_sparse_attn), each with its own queries, reusing the cache and indices.

Default workload: 8-query verify chunk per sequence, batch 4, 131072-token
context, 32 query / 4 KV heads, head_dim 128, top-k 4096 + window 256,
1 full + 3 sparse layers (bf16 cache, fp32 accumulation).

Caches: by default the KV cache is rotated over several identical copies on
the device (at least 4, and at least 2 GiB in all), one copy per step in
turn, so no step finds its cache in the 256 MB memory-side cache or the L2
from an earlier step (a real decode step runs the model's other layers
between two calls of this block).  --caches flush reads a 1 GiB buffer
before every step instead; --caches warm replays one copy.

Cache layout: by default K and V of a token sit side by side, one 2 D
record per (sequence, KV head, token), passed to the library as two
strided views; --kv-layout split allocates K and V as two [B, Hkv, T, D]
tensors (whose distance is then a large power of two at these sizes).

Prints one JSON line (rank 0, N = 1).  Extra fields: achieved algorithmic
GB/s of the step, the roofline of the dominant kernel (full-attention split
kernel) from HIP events around its launches, the measured streaming-read
and gather ceilings of the device (hs2_stream_read_probe), the sparse
layer's roofline against the gather ceiling, per-kernel averages,
per-step percentiles, and the CPU oracle timed on a bounded sample of the
same workload (all host threads, and one thread).
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
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="budget of the oracle sample (half all threads, half one thread)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sa-sink-gate", action="store_true",
                    help="sparse layers with per-head sink logits and sigmoid output gates (hs2_sparse_attn_ex)")
    ap.add_argument("--kv", choices=("bf16", "fp8"), default="bf16",
                    help="cache format: bf16, or OCP E4M3 bytes with one scale per KV head (the _fp8 entry points)")
    ap.add_argument("--block", type=int, default=0,
                    help="block-level selection with blocks of this many tokens (hs2_full_attn_score_select_blocks)")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step in a HIP graph and time its replays (no per-kernel host launches)")
    ap.add_argument("--caches", choices=("rotate", "flush", "warm"), default="rotate",
                    help="rotate: a different copy of the KV cache every step (default); flush: read a 1 GiB buffer "
                         "before every step (timed one by one); warm: the same cache every step")
    ap.add_argument("--kv-layout", choices=("interleaved", "split"), default="interleaved",
                    help="interleaved: K and V of a token in one 2 D record (default); split: two [B, Hkv, T, D] tensors")
    ap.add_argument("--kv-copies", type=int, default=0,
                    help="copies of the KV cache to rotate over (default: at least 4 and at least 2 GiB)")
    ap.add_argument("--stream-probe", action="store_true",
                    help="only measure the streaming-read ceiling (hs2_stream_read_probe) and print it")
    ap.add_argument("--no-stream-probe", action="store_true", help="leave the streaming-read probe out of the line")
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


STREAM_PROBE_BYTES = 4 << 30
GATHER_PROBE_MODES = {512: 4, 256: 5}  # record bytes -> probe mode (scattered-order gathers)
STREAM_PROBE_MODES = {0: "register loads", 1: "register loads, non-temporal", 2: "direct-to-LDS loads",
                      3: "direct-to-LDS loads, non-temporal"}


def stream_probe(dev, reps: int = 8) -> dict:
    """Streaming-read ceiling of the device: hs2_stream_read_probe over a
    4 GiB buffer (16x the memory-side cache) in each load mode; the median of
    `reps` timed launches per mode, the best mode's rate as the ceiling."""
    import torch
    from paper_2609_26368_amd import hs2
    buf = torch.empty(STREAM_PROBE_BYTES // 4, dtype=torch.int32, device=dev)
    buf.random_()
    sink = torch.zeros(hs2.STREAM_PROBE_SINK_WORDS, dtype=torch.int32, device=dev)
    st = torch.cuda.current_stream()
    rates = {}
    for mode in STREAM_PROBE_MODES:
        for _ in range(2):
            hs2.hs2_stream_read_probe(buf, mode, sink, st)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a_, b_ in ev:
            a_.record(st)
            hs2.hs2_stream_read_probe(buf, mode, sink, st)
            b_.record(st)
        torch.cuda.synchronize()
        ms = float(np.median([a_.elapsed_time(b_) for a_, b_ in ev]))
        rates[mode] = STREAM_PROBE_BYTES / (ms * 1e-3) / 1e9
    best = max(rates, key=rates.get)
    # the gather ceilings: the same buffer as records of 512 or 256 bytes
    # (a token's K and V in a bf16 or E4M3 cache of head dim 128) read once
    # each in a scattered order (the sparse layers' access pattern)
    gather = {}
    for rec, mode in GATHER_PROBE_MODES.items():
        for _ in range(2):
            hs2.hs2_stream_read_probe(buf, mode, sink, st)
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a_, b_ in ev:
            a_.record(st)
            hs2.hs2_stream_read_probe(buf, mode, sink, st)
            b_.record(st)
        torch.cuda.synchronize()
        gather[rec] = STREAM_PROBE_BYTES / (float(np.median([a_.elapsed_time(b_) for a_, b_ in ev])) * 1e-3) / 1e9
    del buf
    torch.cuda.empty_cache()
    return {"stream_peak_gbps": round(rates[best], 1), "mode": STREAM_PROBE_MODES[best],
            "gbps_by_mode": {STREAM_PROBE_MODES[m]: round(r, 1) for m, r in rates.items()},
            "gather_gbps_by_record_bytes": {r: round(g, 1) for r, g in gather.items()},
            "bytes": STREAM_PROBE_BYTES, "launches_per_mode": reps}


def kv_copies_for(kv_bytes: int, caches: str, requested: int) -> int:
    """Copies of the KV cache the step rotates over: at least 4 and at least
    2 GiB together (so that no step finds its cache in the 256 MB
    memory-side cache), at most 1024; one when the caches are not rotated."""
    if caches != "rotate":
        return 1
    if requested > 0:
        return requested
    return int(min(1024, max(4, -(-(2 << 30) // max(1, kv_bytes)))))


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
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.stream_probe:
        print(json.dumps(stream_probe(dev)), flush=True)
        return
    probe = None if args.no_stream_probe else stream_probe(dev)
    if probe:
        log(f"[bench] streaming-read probe: {probe['stream_peak_gbps']} GB/s ({probe['mode']}); {probe['gbps_by_mode']}")
    w = W.WORKLOADS[args.workload]
    t = time.perf_counter()
    inp = W.make_inputs(w, kv=args.kv)
    log(f"[bench] inputs {w.name} ({args.kv} cache) generated in {time.perf_counter() - t:.1f}s lens={inp.lens.tolist()}")
    B, C, Hq, Hkv, D = w.batch, w.n_queries, w.n_q_heads, w.n_kv_heads, w.head_dim
    Lmax = inp.K.shape[2]

    def to_dev(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    if args.kv == "fp8":
        K, V = torch.from_numpy(inp.K).to(dev), torch.from_numpy(inp.V).to(dev)
        kv_scales = (torch.from_numpy(inp.k_scale).to(dev), torch.from_numpy(inp.v_scale).to(dev))
    else:
        K, V = to_dev(inp.K), to_dev(inp.V)
        kv_scales = None
    kv_bytes = K.numel() * K.element_size() + V.numel() * V.element_size()
    n_copies = kv_copies_for(kv_bytes, args.caches, args.kv_copies)
    if args.kv_layout == "interleaved":  # one [B, Hkv, T, 2 D] tensor: K in the first D of each record, V after it
        kv_strides = (Hkv * Lmax * 2 * D, Lmax * 2 * D, 2 * D)
        records = [torch.cat([K, V], dim=-1).contiguous()]
        del K, V
        records += [records[0].clone() for _ in range(n_copies - 1)]
        caches = [(r[..., :D], r[..., D:]) for r in records]
    else:
        kv_strides = None
        caches = [(K, V)] + [(K.clone(), V.clone()) for _ in range(n_copies - 1)]
    log(f"[bench] caches: {args.caches}, {n_copies} KV cop{'y' if n_copies == 1 else 'ies'} of {kv_bytes / 1e9:.3f} GB")
    q_fa = to_dev(inp.q_fa)
    q_sa = [to_dev(x) for x in inp.q_sa]
    lens = torch.from_numpy(inp.lens).to(dev)
    blk = hs2.HybridBlock(B, C, Hq, Hkv, D, Lmax, w.k, w.window, device=dev, kv_strides=kv_strides)
    out = torch.empty((B, C, Hq, D), dtype=torch.bfloat16, device=dev)
    idx = torch.empty((B, Hkv, C, w.slots), dtype=torch.int32, device=dev)
    sa_out = [torch.empty_like(out) for _ in q_sa]
    stream = torch.cuda.current_stream()
    sinks, gates = [None] * len(q_sa), [None] * len(q_sa)
    if args.sa_sink_gate:  # synthetic per-layer sink logits and gate logits
        g = torch.Generator(device="cpu").manual_seed(2609)
        sinks = [torch.randn(Hq, generator=g).to(dev) for _ in q_sa]
        gates = [torch.randn((B, C, Hq, D), generator=g).to(torch.bfloat16).to(dev) for _ in q_sa]

    def step_on(st, kv):
        Kc, Vc = kv
        blk.full(q_fa, Kc, Vc, lens, out=out, idx=idx, stream=st, kv_scales=kv_scales, block=args.block)
        for qs, o, sk, gt in zip(q_sa, sa_out, sinks, gates):
            blk.sparse(qs, Kc, Vc, lens, idx, out=o, stream=st, sink=sk, gate=gt, kv_scales=kv_scales)

    n_step = [0]

    def step():  # the next copy of the cache in turn
        step_on(stream, caches[n_step[0] % n_copies])
        n_step[0] += 1

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} steps done")
    run_step = step
    if args.graph:  # one graph per cache copy, captured after the warmup (the library's set-up is done by then)
        graphs = []
        cap = torch.cuda.Stream()
        cap.wait_stream(stream)
        for kv in caches:
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=cap):
                step_on(cap, kv)
            graphs.append(gr)
        torch.cuda.synchronize()

        def run_step():
            graphs[n_step[0] % n_copies].replay()
            n_step[0] += 1
    tokens = B * C
    # flush: evicting by reading 1 GiB (a write would leave dirty lines whose
    # write-back then overlaps the timed step); the read is outside the step's events
    flush = torch.ones(1 << 28, dtype=torch.int32, device=dev) if args.caches == "flush" else None
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall = ev_ms = None
    if flush is None:
        # the timed steps: back to back between one event pair (no marker
        # between steps: on this stack an event record costs a few us of GPU
        # time, which at the 4K decode shape is ~12 % of a step)
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
    # single-step times: a second run of as many steps with an event pair
    # around each (percentiles, the first step after a synchronisation; with
    # --caches flush these are the timed steps, the flush reads outside them)
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    first_copy = n_step[0]
    torch.cuda.synchronize()
    for a_, b_ in ev:
        if flush is not None:
            flush.amax()
        a_.record(stream)
        run_step()
        b_.record(stream)
    torch.cuda.synchronize()
    per_step = np.array([a_.elapsed_time(b_) for a_, b_ in ev])
    if flush is not None:
        ms_per_step = float(per_step.mean())
        value = tokens / (ms_per_step * 1e-3)
        log(f"[bench] timed {args.steps} steps one by one (flushed): mean {ms_per_step:.4f} ms")
    else:
        log(f"[bench] timed {args.steps} steps: wall {wall * 1e3:.2f} ms, events {ev_ms:.2f} ms; "
            f"single steps (second run) sum to {per_step.sum():.2f} ms")
    if n_copies > 1:  # step i of the single-step run used copy (first_copy + i) % n_copies
        by_copy = {}
        for i, ms in enumerate(per_step):
            by_copy.setdefault((first_copy + i) % n_copies, []).append(ms)
        log("[bench] mean step ms by cache copy: " +
            " ".join(f"{c}:{np.mean(v):.4f}" for c, v in sorted(by_copy.items())[:8]))
    pct = {f"p{q}": round(float(np.percentile(per_step, q)), 4) for q in (10, 50, 90)}
    pct["mean"] = round(float(per_step.mean()), 4)
    pct["first"] = round(float(per_step[0]), 4)

    # per-kernel durations (HIP events recorded by the library around each launch, same stream)
    hs2.hs2_timing_enable(True)
    hs2.hs2_timing_reset()
    for _ in range(args.steps):
        if flush is not None:
            flush.amax()
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
    if probe:
        roofline["stream_peak"] = probe["stream_peak_gbps"]
        roofline["frac_of_stream_peak"] = round(achieved / probe["stream_peak_gbps"], 4)
    # the sparse layer: the unique selected rows of each (sequence, KV head)
    # read once, against the gather ceiling
    sa_bytes = uniq * kv_row
    sa_achieved = sa_bytes / (kernels["sa_split"]["avg_us"] * 1e-6) / 1e9
    sa_roofline = {"kernel": "sa_split", "bound": "hbm (gathers)", "achieved": round(sa_achieved, 1),
                   "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(sa_achieved / HBM_PEAK_GBS, 4),
                   "algorithmic_bytes_per_launch": int(sa_bytes)}
    if probe:  # the probe's records closest to this cache's (records of 1 KB: the 512-byte figure)
        rec = 256 if kv_row <= 256 else 512
        gpk = probe["gather_gbps_by_record_bytes"][rec]
        sa_roofline.update({"gather_peak": gpk, "gather_record_bytes": rec,
                            "frac_of_gather_peak": round(sa_achieved / gpk, 4)})

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, inp, args.cpu_seconds)

    cache_desc = {"rotate": f"KV cache rotated over {n_copies} copies ({n_copies * kv_bytes / 1e9:.2f} GB): "
                            f"no step finds its cache in the memory-side cache or L2",
                  "flush": "1 GiB read before every step (outside its events)",
                  "warm": "the same KV cache every step"}[args.caches]
    rec = {"metric": METRIC, "value": round(value, 2), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": w.name, "batch": B, "ctx": w.ctx, "ctx_min": w.ctx_min or w.ctx,
                      "queries_per_seq": C, "q_heads": Hq, "kv_heads": Hkv, "head_dim": D, "k": w.k,
                      "window": w.window, "sparse_layers": w.n_sparse, "needles": w.needles,
                      "kv_cache": "e4m3" if args.kv == "fp8" else "bf16",
                      "kv_layout": ("K and V interleaved: one 2 D record per (sequence, KV head, token)"
                                    if args.kv_layout == "interleaved" else "K and V in two [B, Hkv, T, D] tensors"),
                      "selection": f"block{args.block}" if args.block else "token",
                      "launch": "graph" if args.graph else "eager",
                      "caches": cache_desc,
                      **({"sa_sink_gate": True} if args.sa_sink_gate else {})},
           "achieved_gbps": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
           "algorithmic_bytes_per_step": int(step_bytes),
           "roofline": roofline,
           "sa_roofline": sa_roofline,
           "stream_peak_gbps": probe["stream_peak_gbps"] if probe else None,
           "stream_probe": probe,
           "step_ms_percentiles": pct,
           "kernels_avg_us": {k: round(v["avg_us"], 2) for k, v in kernels.items()},
           "cpu_baseline": cpu}
    print(json.dumps(rec), flush=True)


def cpu_model() -> str:
    """Host CPU model name (the 'model name' line lscpu reports), or ''."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def _oracle_rate(w, inp, budget_s: float):
    """Run the oracle on (sequence, KV head) groups of the inputs, cycling over
    the step's groups, until the budget is spent; returns (tokens/s of whole
    steps, group evaluations, seconds)."""
    from oracle import hs2_oracle as O
    groups_all = [(b, g) for b in range(w.batch) for g in range(w.n_kv_heads)]
    n, t0 = 0, time.perf_counter()
    while True:
        O.hybrid_block(inp.q_fa, inp.q_sa, inp.K, inp.V, inp.lens, w.k, w.window,
                       groups=[groups_all[n % len(groups_all)]], k_scale=inp.k_scale, v_scale=inp.v_scale)
        n += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    step_s = el * len(groups_all) / n
    return w.batch * w.n_queries / step_s, n, el


def cpu_baseline(w, inp, budget_s: float) -> dict:
    """The oracle on (sequence, KV head) groups of the same inputs until the
    budget is spent, scaled to tokens/s of whole steps: once with every BLAS
    thread the host offers, once pinned to one thread (half the budget each)."""
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:  # noqa: BLE001
        threadpool_limits, threads = None, 1
    groups = w.batch * w.n_kv_heads
    v_all, n_all, el_all = _oracle_rate(w, inp, budget_s / 2)
    log(f"[bench] oracle, {threads} threads: {n_all} group evaluations ({groups} per step) in {el_all:.1f}s")
    if threadpool_limits is not None:
        with threadpool_limits(limits=1):
            v_one, n_one, el_one = _oracle_rate(w, inp, budget_s / 2)
    else:
        v_one, n_one, el_one = v_all, n_all, el_all
    log(f"[bench] oracle, 1 thread: {n_one} group evaluations in {el_one:.1f}s")
    return {"value": round(v_all, 4), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{n_all} (sequence, KV head) group evaluations, cycling over the {groups} groups of one "
                      f"step, full context, {el_all:.1f}s; scaled by {groups}/{n_all}",
            "cpu_model": cpu_model(), "cpu_count": os.cpu_count(),
            "single_thread": {"value": round(v_one, 4), "unit": "tokens/s", "cores": 1,
                              "sample": f"{n_one} group evaluations, {el_one:.1f}s, BLAS pinned to one thread"}}


if __name__ == "__main__":
    main()

#!/usr/bin/env python3
"""Benchmark of the EMU Split/Merge reshard on one MI355X.

One step is one pass of the whole hot path over the 8B decoder's state (Llama-3.1-8B shapes, bf16,
synthetic seeded weights): reshard TP2 PP2 -> TP4 PP1 (all 4 source and 4 destination shard sets
resident in HBM), pack the destination shards into 2^28-byte contiguous buckets, and unpack the
buckets into a second, receiver-side destination set. The copy map is compiled once before timing
(its compile time is reported separately). Inputs are resident in HBM before the timed region.

Prints one JSON line. ``value`` is the step's HBM traffic rate: algorithmic bytes read + written by the
three kernels (2 x destination bytes each) divided by the step time. Per-kernel times come from HIP
events recorded on the stream the kernels run on. The ``cpu_baseline`` leg times the CPU oracle on a
bounded sample of the same workload (embedding + the first 16 layers).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
EIGHT_B = (32, 4096, 32, 128, 8, 14336, 128256)  # L, H, nH, hd, G, I, V
TINY = (2, 256, 4, 64, 2, 688, 1024)
ONE_B = (16, 2048, 32, 64, 8, 8192, 128256)
PMC_SUMMARY = os.path.join(ROOT, "profiles", "reshard_8b_tp2pp2_tp4pp1_pmc.txt")
KERNEL_SRCS = [os.path.join(ROOT, "paper_2609_34645_amd", "csrc", f)
               for f in ("emu_exec.hip", "emu_internal.h", "emu_plan.cpp")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def code_only(text):
    """Source text without // comments and blank lines, so that edits to comments keep the hash."""
    lines = (line.split("//", 1)[0].rstrip() for line in text.splitlines())
    return "\n".join(line for line in lines if line)


def kernel_hash(texts=None):
    """Hash of the code that decides the kernels' HBM traffic: the kernels and the plan compiler that
    lays out their tiles and tables (comments excluded)."""
    if texts is None:
        texts = [open(p).read() for p in KERNEL_SRCS]
    return hashlib.sha256("\n".join(code_only(t) for t in texts).encode()).hexdigest()[:16]


def measured_traffic():
    """HBM bytes per reshard launch from the committed rocprofv3 --pmc summary, if it was taken on the
    current kernel source; else None."""
    if not os.path.exists(PMC_SUMMARY):
        return None
    vals = {}
    with open(PMC_SUMMARY) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_code_sha256_16") != kernel_hash():
        return None
    try:
        return float(vals["reshard_hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(seed, layers, bucket_bytes, min_seconds=10.0):
    """Time the CPU oracle on the bench step for a bounded sample: the embedding + the first `layers`
    layers of the same transition, resharded (oracle.reshard_group per tensor group), then each
    destination rank's part of the sample packed into buckets and unpacked (oracle.pack/unpack).
    Repeated passes until at least `min_seconds`, once on one thread and once with a thread pool
    (tensor groups, then ranks) on every host core this process may use; NumPy releases the GIL in its
    copies. Algorithmic bytes as on the GPU: 2 x destination bytes for each of the three steps."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    import oracle

    m = oracle.Model(*EIGHT_B)
    src, dst = oracle.Layout(m, 2, 2), oracle.Layout(m, 4, 1)
    groups = ["embed"] + list(range(layers))
    rng = np.random.default_rng(seed)
    shards = {}
    for r, specs in enumerate(oracle.rank_inventory(src)):
        for j, s in enumerate(specs):
            g = "embed" if s.kind == "embed" else ("final" if s.kind in ("final_norm", "lm_head") else s.layer)
            if g in groups:
                shards[(r, j)] = rng.integers(0, 1 << 16, size=s.shape, dtype=np.uint16)

    def reshard(g):
        return oracle.reshard_group(lambda r, j: shards[(r, j)], src, dst, g)

    def pack_unpack(tensors):
        buckets = oracle.pack(tensors, bucket_bytes)
        back = oracle.unpack(buckets, tensors)
        return sum(a.nbytes for a in back)

    def one_pass(mapper):
        out = {}
        for part in mapper(reshard, groups):
            out.update(part)
        by_rank = {}
        for (r, j) in sorted(out):
            by_rank.setdefault(r, []).append(out[(r, j)])
        moved = sum(a.nbytes for a in out.values())
        assert sum(mapper(pack_unpack, [by_rank[r] for r in sorted(by_rank)])) == moved
        return 6 * moved

    def timed(mapper):
        t = time.perf_counter()
        passes, alg = 0, 0
        while passes < 1 or (time.perf_counter() - t < min_seconds and passes < 50):
            alg += one_pass(mapper)
            passes += 1
        return time.perf_counter() - t, passes, alg

    dt1, p1, a1 = timed(lambda f, xs: [f(x) for x in xs])
    cores = len(os.sched_getaffinity(0))
    with ThreadPoolExecutor(max_workers=cores) as pool:
        dtn, pn, an = timed(lambda f, xs: list(pool.map(f, xs)))
    per_pass = a1 // p1
    return {"value": round(an / dtn / 1e9, 3), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "seconds": round(dtn, 3), "passes": pn, "algorithmic_bytes_per_pass": per_pass,
            "single_thread": {"value": round(a1 / dt1 / 1e9, 3), "cores": 1, "seconds": round(dt1, 3),
                              "passes": p1},
            "host_cpu_count": os.cpu_count(),
            "sample": f"the bench step on the embedding + layers 0-{layers - 1} of the 8B decoder: TP2PP2->TP4PP1 "
                      f"reshard ({per_pass / 6 / 1e9:.2f} GB of destination shards), then each destination rank's "
                      f"part packed into {bucket_bytes}-byte buckets and unpacked; repeated for at least "
                      f"{min_seconds:.0f} s; NumPy, work spread over a pool of {cores} threads (single_thread: "
                      f"one thread); input generation excluded"}


def tiny_latency(emu, iters=200):
    """Latency of the tiny decoder's Split TP1 PP1 -> TP2 PP1 with pack and unpack into 64 KiB buckets
    (3.95 MB of destination shards, cache-resident): back-to-back eager calls through the binding, and
    replays of one HIP graph holding the same three calls. Mean per step over `iters` steps."""
    import torch

    m = emu.Model(*TINY)
    plan = emu.Plan(emu.Layout(m, 1, 1), emu.Layout(m, 2, 1))
    ws = plan.workspace()
    S, D, R = plan.alloc(0, fill=1), plan.alloc(1), plan.alloc(1)
    B = 1 << 16
    bufs, bptrs = plan.alloc_buckets(1, B)

    def step():
        plan.reshard(ws, S.ptrs, D.ptrs)
        plan.pack(ws, 1, B, D.ptrs, bptrs)
        plan.unpack(ws, 1, B, bptrs, R.ptrs)

    def timed(fn):
        for _ in range(10):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / iters

    eager = timed(step)
    cap = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=cap):
        step()
    replay = timed(graph.replay)
    # ten steps in one graph: the graph launch's host cost spread over ten steps, close to the device
    # time of a step (three dependent kernels and the gaps between them)
    graph10 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph10, stream=cap):
        for _ in range(10):
            step()
    replay10 = timed(graph10.replay) / 10
    ok = all(torch.equal(x, y) for x, y in zip(D.tensors, R.tensors))
    # the transport path proper: the sender reshards straight into its buckets (fused plan), the
    # receiver unpacks them; two kernels instead of three
    fused = emu.Plan(plan.src, plan.dst, bucket_bytes=B)
    wf = fused.workspace()
    fbufs, fbptrs = plan.alloc_buckets(1, B)
    R2 = plan.alloc(1)

    def fstep():
        fused.reshard(wf, S.ptrs, fbptrs)
        plan.unpack(ws, 1, B, fbptrs, R2.ptrs)

    f_eager = timed(fstep)
    fgraph10 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(fgraph10, stream=cap):
        for _ in range(10):
            fstep()
    f_replay10 = timed(fgraph10.replay) / 10
    ok = ok and all(torch.equal(x, y) for x, y in zip(D.tensors, R2.tensors))
    # the same path with the receiver's own plan (buckets -> tensors on the reshard kernel)
    recv = emu.Plan(plan.dst, plan.dst, src_bucket_bytes=B)
    wr = recv.workspace()
    R3 = plan.alloc(1)

    def rstep():
        fused.reshard(wf, S.ptrs, fbptrs)
        recv.reshard(wr, fbptrs, R3.ptrs)

    r_eager = timed(rstep)
    rgraph10 = torch.cuda.CUDAGraph()
    with torch.cuda.graph(rgraph10, stream=cap):
        for _ in range(10):
            rstep()
    r_replay10 = timed(rgraph10.replay) / 10
    ok = ok and all(torch.equal(x, y) for x, y in zip(D.tensors, R3.tensors))
    return {"workload": "tiny decoder bf16 TP1PP1->TP2PP1 + pack/unpack at 64 KiB buckets",
            "destination_bytes": plan.info["bytes_written"], "eager_us_per_step": round(eager, 2),
            "graph_us_per_step": round(replay, 2), "graph_of_10_steps_us_per_step": round(replay10, 2),
            "fused_to_buckets_then_unpack": {"eager_us_per_step": round(f_eager, 2),
                                             "graph_of_10_steps_us_per_step": round(f_replay10, 2)},
            "fused_to_buckets_then_receiver_plan": {"eager_us_per_step": round(r_eager, 2),
                                                    "graph_of_10_steps_us_per_step": round(r_replay10, 2)},
            "outputs_consistent": ok}


def variant_timings(emu, seed, reps=5):
    """Mean launch time of the layout variants on the 8B decoder (bf16), each on fresh buffers:
    the paper's T_sub route (TP4 PP8 -> TP4 PP2 -> TP8 PP2, section 6.1) against the direct
    destination-driven TP4 PP8 -> TP8 PP2, and KV replication with uneven stages (TP2 PP2 -> TP16 PP3)."""
    import torch

    from synthetic import device_fill

    model = emu.Model(*EIGHT_B)

    def run(chain):
        plans = [emu.Plan(a, b) for a, b in chain]
        wss = [p.workspace() for p in plans]
        sets = [plans[0].alloc(0)] + [p.alloc(1) for p in plans]
        device_fill(sets[0].tensors, seed, ["norm" if d["kind"].endswith("norm") else "weight"
                                            for d in plans[0].tensors(0)], "bf16")

        def once():
            for p, w, x, y in zip(plans, wss, sets, sets[1:]):
                p.reshard(w, x.ptrs, y.ptrs)

        once()
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        e[0].record()
        for k in range(reps):
            once()
            e[k + 1].record()
        torch.cuda.synchronize()
        ms = sum(e[k].elapsed_time(e[k + 1]) for k in range(reps)) / reps
        moved = sum(p.info["bytes_read"] + p.info["bytes_written"] for p in plans)
        last = sets[-1]
        del sets, wss
        torch.cuda.empty_cache()
        return ms, moved, last, plans[-1]

    L = lambda tp, pp, **kw: emu.Layout(model, tp, pp, **kw)
    out = {}
    d_ms, d_b, d_out, _ = run([(L(4, 8), L(8, 2))])
    t_ms, t_b, t_out, _ = run([(L(4, 8), L(4, 2)), (L(4, 2), L(8, 2))])
    same = all(torch.equal(a, b) for a, b in zip(d_out.bufs, t_out.bufs))
    del d_out, t_out
    torch.cuda.empty_cache()
    out["tsub_route_tp4pp8_to_tp8pp2"] = {
        "direct_ms": round(d_ms, 4), "direct_GBps": round(d_b / (d_ms * 1e-3) / 1e9, 1),
        "via_tp4pp2_ms": round(t_ms, 4), "via_tp4pp2_bytes_over_direct": round(t_b / d_b, 3),
        "outputs_equal": same}
    for name, a, b in (("kv_replication_tp2pp2_to_tp16pp3", L(2, 2), L(16, 3)),):
        ms, moved, _, _ = run([(a, b)])
        out[name] = {"ms": round(ms, 4), "GBps": round(moved / (ms * 1e-3) / 1e9, 1)}
    return out


def bench_other_config(args, emu, torch, cfg):
    """The other workloads, one step each, timed like the default line:
    1 tiny bf16: Split TP1 PP1 -> TP2 PP1 and Merge back (cache-resident: latency);
    2 1B bf16: TP4 PP1 -> TP2 PP1;
    4 8B fp32 training state (master, Adam m, Adam v): TP4 PP1 -> TP1 PP1 as one launch over the three
      tensor groups (emu_reshard_groups), then split back, again one launch; the same two transitions as
      one launch per group are timed beside it, interleaved, on the same buffers;
    5 8B bf16, vocabulary padded to a multiple of 128 per TP rank: TP8 PP4 -> TP2 PP2, pack into
      2^28-byte buckets, unpack into a receiver set."""
    from synthetic import device_fill

    def dists(plan, side):
        return ["norm" if d["kind"].endswith("norm") else "weight" for d in plan.tensors(side)]

    def moved(plan, groups=1):
        return groups * (plan.info["bytes_read"] + plan.info["bytes_written"])

    calls = []        # (name, algorithmic bytes, fn) in step order, the dominant one first
    extra = {}
    keep = []
    if cfg in (1, 2):
        shape, a, b = (TINY, (1, 1), (2, 1)) if cfg == 1 else (ONE_B, (4, 1), (2, 1))
        m = emu.Model(*shape)
        fwd = emu.Plan(emu.Layout(m, *a), emu.Layout(m, *b))
        S, D = fwd.alloc(0), fwd.alloc(1)
        device_fill(S.tensors, args.seed, dists(fwd, 0), "bf16")
        wf = fwd.workspace()
        calls.append(("reshard", moved(fwd), lambda: fwd.reshard(wf, S.ptrs, D.ptrs)))
        if cfg == 1:
            back = emu.Plan(emu.Layout(m, *b), emu.Layout(m, *a))
            wb = back.workspace()
            A2 = back.alloc(1)
            calls.append(("reshard back", moved(back), lambda: back.reshard(wb, D.ptrs, A2.ptrs)))
            keep.append(A2)
        keep += [S, D]
        workload = ("tiny decoder bf16: Split TP1PP1->TP2PP1, then Merge back" if cfg == 1 else
                    "1B decoder bf16: reshard TP4PP1->TP2PP1")
        model_s = "L2 H256 4x64 heads 2 KV MLP688 V1024" if cfg == 1 else "L16 H2048 32x64 heads 8 KV MLP8192 V128256"
    elif cfg == 4:
        m = emu.Model(*EIGHT_B)
        fwd = emu.Plan(emu.Layout(m, 4, 1, 0, "fp32"), emu.Layout(m, 1, 1, 0, "fp32"))
        back = emu.Plan(emu.Layout(m, 1, 1, 0, "fp32"), emu.Layout(m, 4, 1, 0, "fp32"))
        wf, wb = fwd.workspace(), back.workspace()
        Ss, Ds = [], []
        for gi, dist in enumerate(("weight", "adam_m", "adam_v")):
            S, D = fwd.alloc(0), fwd.alloc(1)
            device_fill(S.tensors, args.seed + gi, [dist] * len(S.tensors), "fp32")
            Ss.append(S)
            Ds.append(D)
        st, dt = emu.group_tables(Ss), emu.group_tables(Ds)
        keep += Ss + Ds + [st, dt]
        calls += [("master+m+v TP4->TP1, one launch", moved(fwd, 3), lambda: fwd.reshard_groups(wf, st, dt)),
                  ("master+m+v TP1->TP4, one launch", moved(back, 3), lambda: back.reshard_groups(wb, dt, st))]

        def per_group(plan, w, xs, ys):
            def run():
                for x, y in zip(xs, ys):
                    plan.reshard(w, x.ptrs, y.ptrs)
            return run

        extra["per_group_launches"] = (per_group(fwd, wf, Ss, Ds), per_group(back, wb, Ds, Ss),
                                       lambda: fwd.reshard_groups(wf, st, dt), lambda: back.reshard_groups(wb, dt, st))
        workload = ("8B training state fp32 (master, Adam m, Adam v): TP4PP1->TP1PP1 and back, each direction one "
                    "launch over the three tensor groups")
        model_s = "L32 H4096 32x128 heads 8 KV MLP14336 V128256"
    elif cfg == 5:
        m = emu.Model(*EIGHT_B)
        plan = emu.Plan(emu.Layout(m, 8, 4, 128), emu.Layout(m, 2, 2))
        ws = plan.workspace()
        S, D, R = plan.alloc(0), plan.alloc(1), plan.alloc(1)
        device_fill(S.tensors, args.seed, dists(plan, 0), "bf16")
        B = args.bucket_bytes
        bufs, bptrs = plan.alloc_buckets(1, B)
        keep += [S, D, R, bufs]
        nb = 2 * plan.bucket_layout(1, B, -1)[1]
        calls += [("reshard", moved(plan), lambda: plan.reshard(ws, S.ptrs, D.ptrs)),
                  ("pack", nb, lambda: plan.pack(ws, 1, B, D.ptrs, bptrs)),
                  ("unpack", nb, lambda: plan.unpack(ws, 1, B, bptrs, R.ptrs))]
        workload = "8B decoder bf16, vocab padded to TP*128: reshard TP8PP4->TP2PP2 + pack into 2^28-byte buckets + unpack"
        model_s = "L32 H4096 32x128 heads 8 KV MLP14336 V128256"
    else:
        raise SystemExit(f"unknown config {cfg}")
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        for _n, _b, fn in calls:
            fn()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(calls) + 1)] for _ in range(args.steps)]
    t0 = time.perf_counter()
    for k in range(args.steps):
        evs[k][0].record()
        for j, (_n, _b, fn) in enumerate(calls):
            fn()
            evs[k][j + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [sorted(e[j].elapsed_time(e[j + 1]) for e in evs) for j in range(len(calls))]
    step_bytes = sum(b for _n, b, _ in calls)
    ms_per_step = wall * 1e3 / args.steps
    r_ms = per[0]
    r_avg = sum(r_ms) / len(r_ms)
    r_bytes = calls[0][1]
    achieved = r_bytes / (r_avg * 1e-3) / 1e9
    props = torch.cuda.get_device_properties(0)
    out = {
        "metric": "reshard HBM GB/s (bytes read+written) and ms per transition, % of HBM peak",
        "value": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 2),
        "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic (seeded device draws: N(0,0.02) weights, 1+N(0,0.02) norms, Adam m N(0,1e-3), "
                "v |N(0,1e-6)|)",
        "config": {"workload": workload, "decoder_shape": model_s, "bytes_per_step": step_bytes,
                   "parallelism": "none (1 GPU holds all ranks' shards)", "config_id": cfg},
        "launches": [{"name": n, "mean_ms": round(sum(t) / len(t), 4), "median_ms": round(t[len(t) // 2], 4),
                      "GBps": round(b / (sum(t) / len(t) * 1e-3) / 1e9, 1)}
                     for (n, b, _), t in zip(calls, per)],
        "roofline": {"bound": "hbm", "kernel": "k_reshard", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": None,
                     "algorithmic_bytes_per_launch": r_bytes},
        "device": {"name": props.name, "cus": props.multi_processor_count,
                   "hbm_GB": round(props.total_memory / 1e9, 1)},
        "seed": args.seed,
        "cpu_baseline": None,
    }
    if "per_group_launches" in extra:
        f3, b3, f1, b1 = extra["per_group_launches"]
        reps = max(3, args.steps // 2)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(reps)]
        torch.cuda.synchronize()
        for k in range(reps):
            for j, fn in enumerate((f3, f1, b3, b1)):
                ev[k][j].record()
                fn()
            ev[k][4].record()
        torch.cuda.synchronize()
        med = lambda j: sorted(e[j].elapsed_time(e[j + 1]) for e in ev)[reps // 2]
        out["one_launch_vs_three"] = {
            "tp4_to_tp1_three_launches_ms": round(med(0), 4), "tp4_to_tp1_one_launch_ms": round(med(1), 4),
            "tp1_to_tp4_three_launches_ms": round(med(2), 4), "tp1_to_tp4_one_launch_ms": round(med(3), 4),
            "note": "interleaved on the same buffers, medians"}
    if cfg == 1:
        out["note"] = "3.95 MB of destination shards: cache-resident and latency-bound; read ms_per_step, not GB/s"
    del keep
    return out


def dag_planning(emu):
    """Host-side transition-DAG planning for four model-stages on 1,024 GPUs (8 per node): rollout
    TP4 -> TP8, reward/reference PP2 -> PP4, actor training PP4 -> PP2 on fewer GPUs, critic training
    DP 64 -> 80 onto the GPUs the actor releases. Median planning time of 20 runs."""
    def s(kind, tp, pp, dp, gpus, ttp, tpp, tdp, tg, state):
        return dict(kind=kind, tp=tp, pp=pp, dp=dp, gpus=list(gpus), tgt_tp=ttp, tgt_pp=tpp, tgt_dp=tdp,
                    tgt_gpus=list(tg), state_bytes=state)
    stages = [s(0, 4, 1, 128, range(512), 8, 1, 64, range(512), 16e9),
              s(1, 4, 2, 32, range(512, 768), 4, 4, 16, range(512, 768), 16e9),
              s(2, 4, 4, 32, range(512), 4, 2, 48, range(384), 64e9),
              s(2, 4, 2, 64, range(512, 1024), 4, 2, 80, range(384, 1024), 64e9)]
    runs = [emu.dag_plan(stages) for _ in range(20)]
    r = runs[0]
    return {"gpus": 1024, "primitives": len(r["nodes"]), "edges": len(r["edges"]),
            "resource_edges": r["n_resource_edges"], "l_tran_s": round(r["l_tran"], 4),
            "plan_ms": round(sorted(x["plan_ms"] for x in runs)[10], 4)}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5],
                    help="workload: 1 tiny, 2 1B, 3 8B (default: the headline line), 4 8B fp32 training state, "
                         "5 8B padded vocabulary with buckets")
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--bucket-bytes", type=int, default=1 << 28)
    ap.add_argument("--seed", type=int, default=1234)
    ap.add_argument("--cpu-layers", type=int, default=16)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--tile-vecs", type=int, default=None)
    ap.add_argument("--xcd-remap", type=int, default=None)
    ap.add_argument("--nontemporal", type=int, default=None)
    ap.add_argument("--lds", type=int, default=None)
    ap.add_argument("--bucket-wg-per-cu", type=int, default=None)
    ap.add_argument("--wg-per-cu", type=int, default=None)
    ap.add_argument("--row-wrap", type=int, default=None)
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the reshard is the local step each rank runs, and the library "
              "has no multi-GPU path. Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_34645_amd import emu
    from synthetic import device_fill

    emu.load()
    for opt, v in ((emu.OPT_TILE_VECS, args.tile_vecs), (emu.OPT_XCD_REMAP, args.xcd_remap),
                   (emu.OPT_NONTEMPORAL, args.nontemporal), (emu.OPT_LDS_STAGING, args.lds),
                   (emu.OPT_BUCKET_WG_PER_CU, args.bucket_wg_per_cu), (emu.OPT_WG_PER_CU, args.wg_per_cu),
                   (emu.OPT_ROW_WRAP, args.row_wrap)):
        if v is not None:
            emu.set_option(opt, v)

    torch.cuda.set_device(0)
    if args.config != 3:
        print(json.dumps(bench_other_config(args, emu, torch, args.config)), flush=True)
        return
    dev = torch.device("cuda", 0)
    props = torch.cuda.get_device_properties(dev)
    model = emu.Model(*EIGHT_B)
    L = lambda tp, pp, **kw: emu.Layout(model, tp, pp, **kw)
    src, dst = L(2, 2), L(4, 1)
    B = args.bucket_bytes
    Bs = B - 2                       # phase-shifted buckets: every bucket starts at another 16-byte phase

    t = time.perf_counter()
    plan = emu.Plan(src, dst)
    plan_ms = (time.perf_counter() - t) * 1e3
    info = plan.info
    log(f"plan: {info['n_segments']} segments, {info['n_tiles']} tiles, {plan_ms:.2f} ms")
    # plans that share the benchmark's memory pages: the identity plan (same destination layout,
    # contiguous copies: the copy ceiling), the same transition into separate q/k/v and gate/up tensors,
    # and the PP-only change TP4 PP2 -> TP4 PP1 with and without aliasing of resident shards
    ident = emu.Plan(dst, dst)
    fmt = emu.Plan(src, L(4, 1, qkv="separate", mlp="separate"))
    pp_copy, pp_alias = emu.Plan(L(4, 2), dst), emu.Plan(L(4, 2), dst, alias=True)

    def region(n):
        return torch.empty(n, dtype=torch.uint8, device=dev)

    src_region = region(max(p.region_bytes(0) for p in (plan, ident, pp_copy)))
    dst_region = region(max(p.region_bytes(1) for p in (plan, fmt)))
    bucket_region = region(max([plan.bucket_region_bytes(1, b) for b in (B, Bs)] + [plan.bucket_region_bytes(0, B)]))
    S, SI, SP = plan.views(0, src_region), ident.views(0, src_region), pp_copy.views(0, src_region)
    D, DF = plan.views(1, dst_region), fmt.views(1, dst_region)
    DA = pp_alias.views(1, dst_region, alias=SP)
    R = plan.alloc(1, dev)
    bufs, bptrs = plan.bucket_views(1, B, bucket_region)
    sbufs, sbptrs = plan.bucket_views(1, Bs, bucket_region)
    ws, wsi, wsf = plan.workspace(dev), ident.workspace(dev), fmt.workspace(dev)
    wpc, wpa = pp_copy.workspace(dev), pp_alias.workspace(dev)
    # the plan's upload into a fresh workspace: host-to-device copy of the host tables, then the kernels
    # that derive the tile map and the stream tables (median wall time to completion of 5)
    wup = region(info["workspace_bytes"])
    ups = []
    for _ in range(5):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        plan.upload(wup)
        torch.cuda.synchronize()
        ups.append((time.perf_counter() - t0) * 1e3)
    upload_ms = sorted(ups)[2]
    sdesc = plan.tensors(0)
    device_fill(S.tensors, args.seed, ["norm" if d["kind"].endswith("norm") else "weight" for d in sdesc], "bf16")
    torch.cuda.synchronize()
    log(f"resident: {(src_region.numel() + dst_region.numel() + bucket_region.numel() + sum(b.numel() for b in R.bufs)) / 1e9:.1f} GB")

    reshard_bytes = info["bytes_read"] + info["bytes_written"]
    _, stream_bytes = plan.bucket_layout(1, B, -1)
    bucket_bytes_rw = 2 * stream_bytes
    step_bytes = reshard_bytes + 2 * bucket_bytes_rw

    def step(ev=None):
        if ev:
            ev[0].record()
        plan.reshard(ws, S.ptrs, D.ptrs)
        if ev:
            ev[1].record()
        plan.pack(ws, 1, B, D.ptrs, bptrs)
        if ev:
            ev[2].record()
        plan.unpack(ws, 1, B, bptrs, R.ptrs)
        if ev:
            ev[3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    r_ms = sorted(e[0].elapsed_time(e[1]) for e in evs)
    p_ms = sorted(e[1].elapsed_time(e[2]) for e in evs)
    u_ms = sorted(e[2].elapsed_time(e[3]) for e in evs)
    mean = lambda x: sum(x) / len(x)
    med = lambda x: x[len(x) // 2]
    ok = all(torch.equal(a, b) for a, b in zip(D.tensors, R.tensors))

    def interleaved(fns, reps=args.steps):
        """Median ms of each callable over `reps` rounds, the callables alternating within a round (one
        stream, HIP events around each launch), so that they share time-varying device state."""
        for fn in fns:
            fn()
        ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
              for _ in fns]
        torch.cuda.synchronize()
        for k in range(reps):
            for j, fn in enumerate(fns):
                ev[j][k][0].record()
                fn()
                ev[j][k][1].record()
        torch.cuda.synchronize()
        return [med(sorted(a.elapsed_time(b) for a, b in e)) for e in ev]

    # copy ceiling: the identity plan reads the same source pages and writes the same destination pages
    id_ms, rs_ms = interleaved([lambda: ident.reshard(wsi, SI.ptrs, D.ptrs), lambda: plan.reshard(ws, S.ptrs, D.ptrs)])
    id_bytes = ident.info["bytes_read"] + ident.info["bytes_written"]
    def persistent(fn):
        # the pack/unpack kernel that finds stream offsets with an on-device wave64 scan of each rank's
        # tensor sizes instead of reading the upload-time chunk map
        def run():
            emu.set_option(emu.OPT_BUCKET_TILES, 0)
            try:
                fn()
            finally:
                emu.set_option(emu.OPT_BUCKET_TILES, 1)
        return run

    # phase-shifted buckets against aligned ones, and the device-scan kernel, on the same bucket pages;
    # the last unpack (phase-shifted) is checked
    pk_a, up_a, pk_d, up_d, pk_s, up_s = interleaved([lambda: plan.pack(ws, 1, B, D.ptrs, bptrs),
                                                      lambda: plan.unpack(ws, 1, B, bptrs, R.ptrs),
                                                      persistent(lambda: plan.pack(ws, 1, B, D.ptrs, bptrs)),
                                                      persistent(lambda: plan.unpack(ws, 1, B, bptrs, R.ptrs)),
                                                      lambda: plan.pack(ws, 1, Bs, D.ptrs, sbptrs),
                                                      lambda: plan.unpack(ws, 1, Bs, sbptrs, R.ptrs)])
    shifted_ok = all(torch.equal(a, b) for a, b in zip(D.tensors, R.tensors))

    # fused sender path: source shards straight into the buckets (one pass instead of reshard + pack)
    fused = emu.Plan(src, dst, bucket_bytes=B)
    wf = fused.workspace(dev)
    (f_ms,) = interleaved([lambda: fused.reshard(wf, S.ptrs, bptrs)])
    for b in R.bufs:
        b.zero_()
    plan.unpack(ws, 1, B, bptrs, R.ptrs)
    torch.cuda.synchronize()
    fused_ok = all(torch.equal(a, b) for a, b in zip(D.tensors, R.tensors))
    fused_bytes = fused.info["bytes_read"] + fused.info["bytes_written"]

    # receiver path: the source ranks' TP2 PP2 streams, packed into 2^28-byte buckets (on the bucket
    # region's pages), resharded straight into TP4 PP1 tensors in one pass
    recv = emu.Plan(src, dst, src_bucket_bytes=B)
    wr = recv.workspace(dev)
    s0bufs, s0ptrs = plan.bucket_views(0, B, bucket_region)
    plan.pack(ws, 0, B, S.ptrs, s0ptrs)
    (rv_ms,) = interleaved([lambda: recv.reshard(wr, s0ptrs, R.ptrs)])
    recv_ok = all(torch.equal(a, b) for a, b in zip(D.tensors, R.tensors))
    recv_bytes = recv.info["bytes_read"] + recv.info["bytes_written"]
    del s0bufs, s0ptrs, wr

    # format change (training -> generation layout of q/k/v and gate/up) against the same transition
    # without it, on the same source and destination pages
    fm_ms, base_ms = interleaved([lambda: fmt.reshard(wsf, S.ptrs, DF.ptrs), lambda: plan.reshard(ws, S.ptrs, D.ptrs)])
    fmt_bytes = fmt.info["bytes_read"] + fmt.info["bytes_written"]
    # resident shards aliased: the PP-only change copies nothing when its shards stay where they are
    pc_ms, pa_ms = interleaved([lambda: pp_copy.reshard(wpc, SP.ptrs, D.ptrs),
                                lambda: pp_alias.reshard(wpa, SP.ptrs, DA.ptrs)])
    alias_ok = all(torch.equal(a, b) for a, b in zip(D.tensors, DA.tensors))

    # weight sync from a training stage to a generation stage: fp32 TP4 PP1 master -> bf16 TP2 PP2
    # (layout change and round-to-nearest-even conversion in one pass)
    sync = emu.Plan(emu.Layout(model, 4, 1, 0, "fp32"), emu.Layout(model, 2, 2, 0, "bf16"))
    wsy = sync.workspace(dev)
    SY = sync.alloc(0, dev)
    device_fill(SY.tensors, args.seed + 1, ["norm" if d["kind"].endswith("norm") else "weight"
                                            for d in sync.tensors(0)], "fp32")
    DY = sync.alloc(1, dev)
    (sync_ms,) = interleaved([lambda: sync.reshard(wsy, SY.ptrs, DY.ptrs)])
    sync_bytes = sync.info["bytes_read"] + sync.info["bytes_written"]
    del SY, DY, wsy

    # the runtime's blit copy of the destination bytes (torch copy_), for reference: not a ceiling
    pairs = [(a, b) for a, b in zip(D.tensors, R.tensors)]
    cev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for a, b in pairs:
        b.copy_(a)
    cev[0].record()
    reps = 5
    for _ in range(reps):
        for a, b in pairs:
            b.copy_(a)
    cev[1].record()
    torch.cuda.synchronize()
    blit_ms = cev[0].elapsed_time(cev[1]) / reps
    blit_bytes = 2 * sum(a.numel() for a, _ in pairs)

    ms_per_step = wall * 1e3 / args.steps
    reshard_avg = mean(r_ms)
    achieved = reshard_bytes / (reshard_avg * 1e-3) / 1e9
    gbps = lambda nbytes, ms: round(nbytes / (ms * 1e-3) / 1e9, 1)
    traffic = measured_traffic()
    out = {
        "metric": "reshard HBM GB/s (bytes read+written) and ms per 8B transition, % of HBM peak",
        "value": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic (seeded N(0,0.02) bf16 weights, 1+N(0,0.02) norms; Llama-3.1-8B shapes)",
        "config": {
            "workload": "8B decoder bf16: reshard TP2PP2->TP4PP1 + pack into 2^28-byte buckets + unpack",
            "decoder_shape": "L32 H4096 32x128 heads 8 KV MLP14336 V128256",
            "src_layout": "TP2PP2", "dst_layout": "TP4PP1", "bucket_bytes": B,
            "bytes_per_step": step_bytes, "parallelism": "none (1 GPU holds all ranks' shards)",
        },
        "reshard_ms": round(reshard_avg, 4),
        "reshard_ms_median": round(med(r_ms), 4),
        "reshard_ms_min_max": [round(r_ms[0], 4), round(r_ms[-1], 4)],
        "reshard_GBps": round(achieved, 1),
        "reshard_pct_of_peak": round(100 * achieved / HBM_PEAK_GBPS, 2),
        "pack_ms": round(mean(p_ms), 4),
        "unpack_ms": round(mean(u_ms), 4),
        "pack_GBps": gbps(bucket_bytes_rw, mean(p_ms)),
        "unpack_GBps": gbps(bucket_bytes_rw, mean(u_ms)),
        "transition_ms": round(reshard_avg + mean(p_ms) + mean(u_ms), 4),
        "identity_copy_ms": round(id_ms, 4),
        "identity_copy_GBps": gbps(id_bytes, id_ms),
        "reshard_interleaved_ms": round(rs_ms, 4),
        "reshard_over_identity": round(rs_ms / id_ms, 4),
        "phase_shifted_bucket_bytes": Bs,
        "pack_aligned_interleaved_ms": round(pk_a, 4),
        "unpack_aligned_interleaved_ms": round(up_a, 4),
        "pack_phase_shifted_ms": round(pk_s, 4),
        "unpack_phase_shifted_ms": round(up_s, 4),
        "pack_phase_shifted_pct_of_peak": round(100 * bucket_bytes_rw / (pk_s * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
        "unpack_phase_shifted_pct_of_peak": round(100 * bucket_bytes_rw / (up_s * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
        "pack_aligned_interleaved_pct_of_peak": round(100 * bucket_bytes_rw / (pk_a * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
        "unpack_aligned_interleaved_pct_of_peak": round(100 * bucket_bytes_rw / (up_a * 1e-3) / 1e9 / HBM_PEAK_GBPS, 2),
        "phase_shifted_outputs_consistent": shifted_ok,
        "pack_device_scan_ms": round(pk_d, 4),
        "unpack_device_scan_ms": round(up_d, 4),
        "fused_reshard_to_buckets_ms": round(f_ms, 4),
        "fused_reshard_to_buckets_GBps": gbps(fused_bytes, f_ms),
        "fused_vs_reshard_plus_pack": round((reshard_avg + mean(p_ms)) / f_ms, 3),
        "fused_outputs_consistent": fused_ok,
        "receiver_reshard_from_buckets_ms": round(rv_ms, 4),
        "receiver_reshard_from_buckets_GBps": gbps(recv_bytes, rv_ms),
        "receiver_outputs_consistent": recv_ok,
        "formats_fused_to_separate_tp2pp2_to_tp4pp1": {
            "ms": round(fm_ms, 4), "GBps": gbps(fmt_bytes, fm_ms), "same_pages_fused_to_fused_ms": round(base_ms, 4),
            "ratio": round(fm_ms / base_ms, 4)},
        "alias_resident_pp_only_tp4pp2_to_tp4pp1": {
            "copy_ms": round(pc_ms, 4), "copy_GBps": gbps(pp_copy.info["bytes_read"] + pp_copy.info["bytes_written"], pc_ms),
            "aliased_ms": round(pa_ms, 4), "aliased_bytes_moved": pp_alias.info["bytes_read"] + pp_alias.info["bytes_written"],
            "alias_tensors": pp_alias.info["n_alias_tensors"], "outputs_equal": alias_ok},
        "weight_sync_fp32_tp4pp1_to_bf16_tp2pp2_ms": round(sync_ms, 4),
        "weight_sync_GBps": gbps(sync_bytes, sync_ms),
        "plan_compile_ms": round(plan_ms, 3),
        "plan_upload_ms": round(upload_ms, 3),
        "workspace_bytes": info["workspace_bytes"],
        "transition_dag_1024_gpus": dag_planning(emu),
        "blit_copy_GBps": gbps(blit_bytes, blit_ms),
        "roofline": {
            "bound": "hbm",
            "kernel": "k_reshard",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": reshard_bytes,
        },
        "options": {k: emu.get_option(v) for k, v in (("tile_vecs", emu.OPT_TILE_VECS),
                                                      ("xcd_remap", emu.OPT_XCD_REMAP),
                                                      ("nontemporal", emu.OPT_NONTEMPORAL),
                                                      ("lds_staging", emu.OPT_LDS_STAGING),
                                                      ("bucket_wg_per_cu", emu.OPT_BUCKET_WG_PER_CU),
                                                      ("bucket_tiles", emu.OPT_BUCKET_TILES),
                                                      ("row_wrap", emu.OPT_ROW_WRAP),
                                                      ("wg_per_cu", emu.OPT_WG_PER_CU))},
        "device": {"name": props.name, "cus": props.multi_processor_count,
                   "hbm_GB": round(props.total_memory / 1e9, 1)},
        "outputs_consistent": ok,
        "seed": args.seed,
    }
    del S, SI, SP, D, DF, DA, R, bufs, sbufs, src_region, dst_region, bucket_region
    torch.cuda.empty_cache()
    out["tiny_transition_latency"] = tiny_latency(emu)
    log("timing the layout variants ...")
    out["variants_8b"] = variant_timings(emu, args.seed)
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(args.seed, args.cpu_layers, B)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

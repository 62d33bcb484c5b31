#!/usr/bin/env python
"""Benchmark of the DominoTree draft-tree builder on one MI355X.

One step = one dt_build_tree call over one batch of resident synthetic logits:
top-M scan, row merge, expansion and emission (every kernel of the path).  The
default workload is the Qwen3-8B-shaped single stream (L=16, V=151936, M=64,
B=16, T=1, d_e=4096, d_h=512).

Timing.  After the warm-up the K calls run once eagerly: per-call GPU times
from torch events, and each kernel's execution time from HIP events the
library takes at the kernel's start and end on its launch stream (every call
when K < 64, else every 8th).  The same K calls are then captured into one HIP
graph, replayed once untimed and checked against the eager pass, and timed as
one replay: `value` = trees/s over that replay's wall clock.  Logit buffers
rotate through >= 512 MB, and a 1 GiB device copy runs between the untimed and
the timed replay, so the timed scan never finds its logits in the 256 MB
Infinity Cache, whatever K is.  A short pass with expansion statistics on then
gives the dependent expansion steps per tree, the expanded nodes and the depth
histogram of the trees built.

The CPU baseline (the oracle as it stands, float64 numpy, one BLAS thread per
worker) runs first, before the GPU is touched: a single-core leg and an
all-core leg over a fork pool of min(nproc, 16) workers, on trees of the same
workload.

Prints ONE JSON line: trees/s for the whole job, the roofline of the dominant
kernel (the expansion at one tree per call: fp32-precision MFMA work, priced
against the fp32 peak; it is a chain of dependent steps, so the line's
`latency` block carries us per dependent step and the occupancy), the scan's
HBM roofline, and the CPU baseline.

--scorer marg|static times the ablation arms; --scorer head times
dt_build_tree_head (Domino's own rank-256 SiLU head over [H_d; S], d_H = d_e,
synthetic hidden states); its stage "expand" is the tree kernel: the expansion
kernel with the head's correction at the Qwen shapes (rank 256 split 16 or 32
per member), else the one-workgroup head kernel.  --max-children k caps the
children of a node (0: the slice, M).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
FP32_PEAK_TFLOPS = 157.3    # dense fp32 (MFMA and vector) of the MI355X
PROFILES = os.path.join(ROOT, "profiles")
SCORERS = {"cond": 0, "marg": 1, "static": 2, "head": 3}
WORKLOADS = ["tiny", "qwen3_4b", "qwen3_8b", "budget64", "concurrent", "deep", "deep_concurrent"]
HEAD_RANK = 256   # the paper's bottleneck rank for Domino's own head
MAX_WORKERS = 16  # CPU share of one GPU on the benchmark box
STATS_CALLS = 32  # calls of the statistics pass


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="qwen3_8b", choices=WORKLOADS)
    ap.add_argument("--rotate-mb", type=float, default=512.0,
                    help="logit bytes cycled through in the timed loop")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="single-core oracle leg; the all-core leg takes about half of it")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--max-children", type=int, default=0,
                    help="children per expanded node (k); 0: all M slots")
    ap.add_argument("--scorer", default="cond", choices=list(SCORERS),
                    help="children function: cond (DominoTree), marg or static (the ablation "
                         "arms), head (Domino's own head)")
    ap.add_argument("--eager", action="store_true",
                    help="time the K calls launched one by one instead of one HIP-graph replay")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 256 MiB device copy (scale for PMC byte counters)")
    return ap.parse_args()


def expansion_flops(cfg, nodes):
    """fp32-precision MFMA work of `nodes` expansions (W_hh . S for the GRU plus
    the slice correction U . S; Domino's own head: W_1^S S and W_2[cand] . y)."""
    dh, M = cfg["d_h"], cfg["M"]
    if cfg.get("rank"):
        return nodes * 2.0 * (3 * dh * dh + cfg["rank"] * (dh + M))
    return nodes * 2.0 * (3 * dh * dh + M * dh)


def source_digest(files):
    """sha256 over the kernel sources a counter record was taken with."""
    import hashlib
    h = hashlib.sha256()
    for f in files:
        h.update(open(os.path.join(ROOT, "paper_2607_08642_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def traffic_from_profiles(workload, stage):
    """HBM bytes per launch from the committed PMC record, if it matches the current kernel."""
    path = os.path.join(PROFILES, "pmc_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))["records"].get(workload, {}).get(stage)
        if not rec or source_digest(rec["sources"]) != rec["sha256"]:
            return None          # no record, or the kernel changed since the counters were taken
        return rec["bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        return None


def cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# ---- CPU baseline: the oracle, one BLAS thread per worker ----------------------
_CPU = {}   # inputs of the oracle legs (inherited by the forked workers)


def _oracle_tree(n):
    import oracle
    c = _CPU
    wl = c["wl"]
    buf = c["bufs"][(n // wl.batch) % len(c["bufs"])]
    t = n % wl.batch
    oracle.build_tree(buf[t], wl.weights.emb, wl.weights.dtype, c["wd"],
                      None if wl.h0 is None else wl.h0[t], wl.M, wl.B, wl.T,
                      max_children=c["k"], logits_dtype=wl.logits_dtype, scorer=c["scorer"],
                      H=None if c["head"] is None else c["head"][1][t])


def _worker(args):
    """Trees built by one pool worker in `seconds` (tree indices start at `first`)."""
    first, stride, seconds = args
    from threadpoolctl import threadpool_limits
    n, t0 = 0, time.perf_counter()
    with threadpool_limits(limits=1):
        while True:
            _oracle_tree(first + n * stride)
            n += 1
            if time.perf_counter() - t0 >= seconds and n >= 2:
                return n, time.perf_counter() - t0


def cpu_baseline(wl_name, wl, bufs_host, seconds, scorer=0, head=None, k=0):
    """The oracle as it stands: a single-core leg, then an all-core fork pool."""
    import multiprocessing as mp
    w = wl.weights
    wd = dict(w_ih=w.w_ih, w_hh=w.w_hh, b_ih=w.b_ih, b_hh=w.b_hh, w_c=w.w_c, b_c=w.b_c,
              dtype=w.dtype)
    if head is not None:
        wd.update(w1=head[0].w1, w2=head[0].w2)
    _CPU.update(wl=wl, bufs=bufs_host, wd=wd, scorer=scorer, head=head, k=k)
    n1, el1 = _worker((0, 1, seconds))
    nproc = os.cpu_count() or 1
    workers = max(1, min(nproc, MAX_WORKERS))
    leg = max(2.0, seconds / 2)
    with mp.get_context("fork").Pool(workers) as pool:
        t0 = time.perf_counter()
        res = pool.map(_worker, [(1000 + i, workers, leg) for i in range(workers)])
        wall = time.perf_counter() - t0
    nall = sum(n for n, _ in res)
    return {"value": nall / wall, "unit": "trees/s", "cores": workers, "kind": "oracle",
            "sample": f"{nall} trees of the {wl_name} workload on {workers} worker processes "
                      f"({wall:.1f} s wall), float64 numpy oracle, 1 BLAS thread each; "
                      f"single core: {n1} trees in {el1:.1f} s",
            "single_core": {"value": n1 / el1, "unit": "trees/s", "cores": 1},
            "nproc": nproc, "cpu_model": cpu_model()}


def head_on_expand(rank, G):
    """Whether dt_build_tree_head runs on the expansion kernel (the library's
    rule: rank a multiple of 16 G with 16, 32 or 64 ranks per member)."""
    return rank % (16 * G) == 0 and rank // G in (16, 32, 64)


def group_size(d_h, num_cus, batch):
    """Workgroups per tree of the expansion kernel (the library's rule): the largest
    power of two <= 16 with >= 32 hidden units (a multiple of 16) per member and
    a grid of at most one workgroup per CU."""
    G = 16
    while G > 1 and (d_h // G < 32 or (d_h // G) % 16 != 0 or 8 * G * ((batch + 7) // 8) > num_cus):
        G //= 2
    return G


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(independent trees would shard across GPUs with no exchange).", file=sys.stderr)
        sys.exit(2)

    import numpy as np

    from paper_2607_08642_amd import synth

    wl = synth.WORKLOADS[args.workload]()
    w = wl.weights
    d = w.dtype
    head = None
    if args.scorer == "head":
        # Domino's own head (dt_build_tree_head): d_H = the drafter's width,
        # rank 256, synthetic hidden states
        hw = synth.domino_head(43, w.V, w.d_e, w.d_h, HEAD_RANK, d, w2_scale=0.5)
        hH = synth.hidden_states(43, wl.batch, wl.L, w.d_e, d)
        head = (hw, hH)
    per_buf = wl.logits.nbytes
    nbuf = max(1, math.ceil(args.rotate_mb * 2**20 / per_buf))
    bufs_host = [wl.logits] + [synth.logits_buffer(wl.name, i, wl.batch) for i in range(1, nbuf)]

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl.name, wl, bufs_host, args.cpu_seconds, SCORERS[args.scorer], head,
                           args.max_children)

    # ---- the GPU from here on -------------------------------------------------
    import torch

    from paper_2607_08642_amd import binding
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")

    def up(a, dt):
        if a is None:
            return None
        if dt == synth.DT_BF16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

    emb = up(w.emb, d)
    plan = binding.Plan(emb, up(w.w_ih, d), up(w.w_hh, d), up(w.b_ih, d), up(w.b_hh, d),
                        up(w.w_c, d), up(w.b_c, d), L=wl.L, M=wl.M, B=wl.B,
                        logits_dtype=wl.logits_dtype, max_batch=wl.batch,
                        max_children=args.max_children,
                        scorer=0 if args.scorer == "head" else SCORERS[args.scorer])
    if head is not None:
        w1, w2, Hdev = up(head[0].w1, d), up(head[0].w2, d), up(head[1], d)
    bufs = [up(b, wl.logits_dtype) for b in bufs_host]
    h0 = None if wl.h0 is None else torch.from_numpy(wl.h0).to(dev)
    out = binding.Tree.empty(wl.batch, wl.B, dev)
    stream = torch.cuda.current_stream()
    if head is None:
        ws = plan.workspace(wl.batch)

        def step(i, o=out):
            plan.build_tree(bufs[i % nbuf], wl.T, h0, out=o, workspace=ws)
    else:
        ws = torch.empty(plan.head_workspace_size(wl.batch, w1, w2), dtype=torch.uint8, device=dev)

        def step(i, o=out):
            plan.build_tree_head(bufs[i % nbuf], Hdev, w1, w2, wl.T, h0, out=o, workspace=ws)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    # eager pass over the K calls: per-call GPU times, and the kernels' own start
    # and end events on the launch stream
    profile_every = 1 if args.steps < 64 else 8
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    plan.set_profiling(profile_every)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        evs[i].record(stream)
        step(args.warmup + i)
    evs[-1].record(stream)
    torch.cuda.synchronize()
    eager_wall = time.perf_counter() - t0
    per_call = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]) * 1e3  # us
    stage_us = {k: v * 1e3 for k, v in plan.stage_ms().items()}  # mean over the profiled calls
    profiled = (args.steps + profile_every - 1) // profile_every
    plan.set_profiling(0)
    eager_last = {k: getattr(out, k).cpu().clone() for k in ("tokens", "parents", "scores", "mask")}

    # a read and a write of 1 GiB: nothing of the logits is left in the caches
    flush_src = torch.empty(2**30 // 4, dtype=torch.float32, device=dev).fill_(1.0)
    flush_dst = torch.empty_like(flush_src)
    if args.eager:
        wall = eager_wall
    else:
        # the same K calls captured into one HIP graph (two kernel nodes per
        # call, no copies or memsets), replayed once untimed, checked against
        # the eager pass, then timed as one replay
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(args.steps):
                step(args.warmup + i)
        graph.replay()
        torch.cuda.synchronize()
        for k, v in eager_last.items():
            if not torch.equal(getattr(out, k).cpu(), v):
                raise RuntimeError(f"graph replay differs from the eager calls in {k}")
        flush_dst.copy_(flush_src)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        graph.replay()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        del graph
    del flush_src, flush_dst

    # statistics pass: expansion steps and expanded nodes per tree (the
    # kernel's own count, speculative expansions included), depth histogram
    steps_tree, exp_tree, steps_call = [], [], []
    dhist = np.zeros(wl.L + 1, np.int64)
    alg_nodes = []
    ncalls = min(STATS_CALLS, nbuf)
    num_cus = torch.cuda.get_device_properties(0).multi_processor_count
    G = group_size(w.d_h, num_cus, wl.batch)
    head_fast = head is not None and head_on_expand(HEAD_RANK, G)
    if head is None or head_fast:
        plan.set_profiling(1)
        for i in range(ncalls):
            step(i)
            st, ex = plan.expand_stats(wl.batch)
            steps_tree += st
            exp_tree += ex
            steps_call.append(max(st))
            dep = out.depth.cpu().numpy()
            nn = out.n_nodes.cpu().numpy()
            for t in range(wl.batch):
                dhist += np.bincount(dep[t, :nn[t]], minlength=wl.L + 1)
                # Alg. 1's expansions: the root plus every popped node above depth L
                alg_nodes.append(int(np.sum(dep[t, :nn[t]] < wl.L)) + 1)
        plan.set_profiling(0)
    else:
        for i in range(ncalls):
            step(i)
            dep = out.depth.cpu().numpy()
            nn = out.n_nodes.cpu().numpy()
            for t in range(wl.batch):
                dhist += np.bincount(dep[t, :nn[t]], minlength=wl.L + 1)
                alg_nodes.append(int(np.sum(dep[t, :nn[t]] < wl.L)) + 1)
    torch.cuda.synchronize()

    cfg = dict(batch=wl.batch, L=wl.L, V=w.V, M=wl.M, d_e=w.d_e, d_h=w.d_h,
               logit_bytes=2 if wl.logits_dtype == synth.DT_BF16 else 4,
               rank=HEAD_RANK if head is not None else 0)
    rows = wl.batch * wl.L
    scan_bytes = rows * w.V * cfg["logit_bytes"]
    scan_us, exp_us = stage_us["scan"], stage_us["expand"]
    # expansions per call Alg. 1 performs (the kernel's speculative extra ones are
    # not counted as useful work)
    alg_per_call = float(np.mean(alg_nodes)) * wl.batch
    exp_flops = expansion_flops(cfg, alg_per_call)
    slow_head = head is not None and not head_fast
    exp_roof = {"kernel": "head_tree" if slow_head else "expand",
                "bound": "alu" if slow_head else "mfma",
                "achieved": exp_flops / (exp_us * 1e-6) / 1e12, "peak": FP32_PEAK_TFLOPS,
                "unit": "TFLOP/s"}
    exp_roof["frac"] = exp_roof["achieved"] / exp_roof["peak"]
    exp_roof["traffic"] = None if head is not None or args.max_children else \
        traffic_from_profiles(wl.name, "expand")
    scan_gbps = scan_bytes / (scan_us * 1e-6) / 1e9
    scan_roof = {"kernel": "scan", "bound": "hbm", "achieved": scan_gbps, "peak": HBM_PEAK_GBS,
                 "unit": "GB/s", "frac": scan_gbps / HBM_PEAK_GBS,
                 "traffic": traffic_from_profiles(wl.name, "scan")}
    dom_is_scan = scan_us > exp_us
    latency = {"expand_us": exp_us, "scan_us": scan_us}
    if steps_call:
        latency.update({
            "steps_per_tree_mean": float(np.mean(steps_tree)),
            "steps_per_call_max_mean": float(np.mean(steps_call)),
            "us_per_step": exp_us / float(np.mean(steps_call)),
            "expanded_nodes_per_tree_mean": float(np.mean(exp_tree)),
            "alg_expansions_per_tree_mean": float(np.mean(alg_nodes)),
            "us_per_pop": exp_us / wl.B,   # per tree: the trees of a call run side by side
            "workgroups_per_tree": G, "grid": (8 * G * ((wl.batch + 7) // 8)) if G > 1 else wl.batch,
            "waves_per_workgroup": 8, "num_cus": num_cus,
            "stats_calls": ncalls,
        })
    trees = wl.batch * args.steps
    res = {
        "metric": "draft trees built/sec",
        "value": trees / wall,
        "unit": "trees/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if d == synth.DT_BF16 else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name if args.scorer == "cond" else f"{wl.name}-{args.scorer}",
                   "scorer": args.scorer, "batch": wl.batch, "L": wl.L, "V": w.V, "M": wl.M,
                   "B": wl.B, "T": wl.T, "d_e": w.d_e, "d_h": w.d_h, "logit_buffers": nbuf},
        "timing": "eager" if args.eager else "hip_graph",
        "us_per_tree": wall / trees * 1e6,
        "eager": {"us_per_tree": eager_wall / trees * 1e6,
                  "gpu_us_per_call_p50": float(np.percentile(per_call, 50)),
                  "gpu_us_per_call_p99": float(np.percentile(per_call, 99))},
        "stages_us": stage_us,
        "stage_calls_profiled": profiled,
        "scan_gbps": scan_gbps,
        "scan_hbm_frac": scan_gbps / HBM_PEAK_GBS,
        "roofline": scan_roof if dom_is_scan else exp_roof,
        "scan_roofline": scan_roof,
        "expand_roofline": exp_roof,
        "latency": latency,
        "depth_hist": dhist.tolist(),
    }
    if head is not None:
        res["config"].update(d_H=w.d_e, rank=HEAD_RANK)
    if args.max_children:
        res["config"]["k"] = args.max_children
        res["config"]["workload"] += f"-k{args.max_children}"
    if args.copy_calibration:
        x = torch.empty(256 * 2**20 // 4, dtype=torch.float32, device=dev).fill_(1.0)
        y = torch.empty_like(x)
        y.copy_(x)
        torch.cuda.synchronize()
    if cpu is not None:
        res["cpu_baseline"] = cpu
    plan.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

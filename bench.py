#!/usr/bin/env python
"""Benchmark of the DominoTree draft-tree builder on one MI355X.

One step = one dt_build_tree call over one batch of resident synthetic logits:
top-M scan, row merge, expansion and emission (every kernel of the path).  The
default workload is the Qwen3-8B-shaped single stream (L=16, V=151936, M=64,
B=16, T=1, d_e=4096, d_h=512).  Logit buffers rotate through >= 512 MB so the
256 MB Infinity Cache cannot serve the scan.

The K timed calls are captured into one HIP graph and timed as one replay
(--eager: launched one by one); the same K calls also run eagerly first, which
gives the per-call GPU times and the stage durations (every 8th call launches
its two kernels with start and end events, so a stage is one kernel's execution
time), and the graph's output is checked against theirs.

Prints ONE JSON line: trees/s for the whole job, the per-kernel roofline of the
dominant kernel and the CPU oracle timed on a bounded sample.

--scorer marg|static times the ablation arms; --scorer head times
dt_build_tree_head (Domino's own rank-256 SiLU head over [H_d; S], d_H = d_e,
synthetic hidden states); its stage "expand" is the head path's tree kernel.
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
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
PROFILES = os.path.join(ROOT, "profiles")
SCORERS = {"cond": 0, "marg": 1, "static": 2, "head": 3}
HEAD_RANK = 256   # the paper's bottleneck rank for Domino's own head
PROFILE_EVERY = 8   # kernel start/end events on every 8th eager call


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="qwen3_8b",
                    choices=["tiny", "qwen3_4b", "qwen3_8b", "budget64", "concurrent"])
    ap.add_argument("--rotate-mb", type=float, default=512.0,
                    help="logit bytes cycled through in the timed loop")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--scorer", default="cond", choices=list(SCORERS),
                    help="children function: cond (DominoTree), marg or static (the ablation arms)")
    ap.add_argument("--eager", action="store_true",
                    help="time the K calls launched one by one instead of one HIP-graph replay")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one plain 256 MiB device copy (scale for PMC byte counters)")
    return ap.parse_args()


def algorithmic(plan_cfg, stage):
    """Algorithmic work of one launch of a stage: (bytes or flops, unit, bound)."""
    c = plan_cfg
    rows = c["batch"] * c["L"]
    if stage == "scan":
        return rows * c["V"] * c["logit_bytes"], "bytes", "hbm"
    # expansion: MFMA work of Alg. 1's expansions (GRU hidden GEMV + slice correction;
    # Domino's own head: W_1^S S and W_2[cand] . y in place of the linear head)
    n = c["expanded_nodes_per_call"]
    if c.get("rank"):
        return n * 2.0 * (3 * c["d_h"] * c["d_h"] + c["rank"] * (c["d_h"] + c["M"])), "flops", "mfma"
    return n * 2.0 * (3 * c["d_h"] * c["d_h"] + c["M"] * c["d_h"]), "flops", "mfma"


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


def cpu_baseline(wl_name, wl, bufs_host, seconds, scorer=0, head=None):
    """The oracle as it stands, one BLAS thread, on trees of the same workload."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    w = wl.weights
    wd = dict(w_ih=w.w_ih, w_hh=w.w_hh, b_ih=w.b_ih, b_hh=w.b_hh, w_c=w.w_c, b_c=w.b_c,
              dtype=w.dtype)
    if head is not None:
        wd.update(w1=head[0].w1, w2=head[0].w2)
    n = 0
    t0 = time.perf_counter()
    with threadpool_limits(limits=1):
        while True:
            buf = bufs_host[(n // wl.batch) % len(bufs_host)]
            t = n % wl.batch
            oracle.build_tree(buf[t], w.emb, w.dtype, wd, None if wl.h0 is None else wl.h0[t],
                              wl.M, wl.B, wl.T, logits_dtype=wl.logits_dtype, scorer=scorer,
                              H=None if head is None else head[1][t])
            n += 1
            el = time.perf_counter() - t0
            if el >= seconds and n >= 3:
                break
    return {"value": n / el, "unit": "trees/s", "cores": 1, "kind": "oracle",
            "sample": f"{n} trees of the {wl_name} workload (first rotation buffers), "
                      f"float64 numpy oracle, 1 BLAS thread, {el:.1f} s"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(independent trees would shard across GPUs with no exchange).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_08642_amd import binding, synth
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")

    wl = synth.WORKLOADS[args.workload]()
    w = wl.weights
    d = w.dtype

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
                        scorer=0 if args.scorer == "head" else SCORERS[args.scorer])
    head = None
    if args.scorer == "head":
        # Domino's own head (dt_build_tree_head): d_H = the drafter's width,
        # rank 256, synthetic hidden states
        hw = synth.domino_head(43, w.V, w.d_e, w.d_h, HEAD_RANK, d, w2_scale=0.5)
        hH = synth.hidden_states(43, wl.batch, wl.L, w.d_e, d)
        head = (hw, hH)
        w1, w2, Hdev = up(hw.w1, d), up(hw.w2, d), up(hH, d)
    per_buf = wl.logits.nbytes
    nbuf = max(1, math.ceil(args.rotate_mb * 2**20 / per_buf))
    bufs_host = [wl.logits] + [synth.logits_buffer(wl.name, i, wl.batch) for i in range(1, nbuf)]
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

    # eager pass over the same K calls: per-call GPU times and the stage
    # events the library records on the launch stream (every PROFILE_EVERY-th call)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    plan.set_profiling(PROFILE_EVERY)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        evs[i].record(stream)
        step(args.warmup + i)
    evs[-1].record(stream)
    torch.cuda.synchronize()
    eager_wall = time.perf_counter() - t0
    per_call = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)]) * 1e3  # us
    stage_us = {k: v * 1e3 for k, v in plan.stage_ms().items()}  # mean over the sampled calls
    plan.set_profiling(0)
    eager_last = {k: getattr(out, k).cpu().clone() for k in ("tokens", "parents", "scores", "mask")}

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
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        graph.replay()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0

    # expansions Alg. 1 performs: the root plus every popped node above depth L
    # (the kernel's extra speculative expansions are not counted as useful work)
    dep = out.depth.cpu().numpy()
    nn = out.n_nodes.cpu().numpy()
    expanded = int(sum(int(np.sum(dep[t, :nn[t]] < wl.L)) + 1 for t in range(wl.batch)))
    rows = wl.batch * wl.L
    cfg = dict(batch=wl.batch, L=wl.L, V=w.V, M=wl.M, d_e=w.d_e, d_h=w.d_h,
               logit_bytes=2 if wl.logits_dtype == synth.DT_BF16 else 4,
               expanded_nodes_per_call=expanded, rank=HEAD_RANK if head is not None else 0)
    scan_bytes = rows * w.V * cfg["logit_bytes"]
    dom = max(stage_us, key=stage_us.get)
    work, unit, bound = algorithmic(cfg, dom)
    dur_s = stage_us[dom] * 1e-6
    if unit == "bytes":
        achieved, peak, runit = work / dur_s / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved = work / dur_s / 1e12
        peak = MFMA_PEAK_TFLOPS["bf16" if d == synth.DT_BF16 else "f32"]
        runit = "TFLOP/s"
    scan_us = stage_us["scan"]
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
    }
    res.update({
        "scan_gbps": scan_bytes / (scan_us * 1e-6) / 1e9,
        "scan_hbm_frac": scan_bytes / (scan_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
        "roofline": {"kernel": dom, "bound": bound, "achieved": achieved, "peak": peak,
                     "unit": runit, "frac": achieved / peak,
                     "traffic": traffic_from_profiles(wl.name, dom)},
        "scan_roofline": {"kernel": "scan", "bound": "hbm",
                          "achieved": scan_bytes / (scan_us * 1e-6) / 1e9,
                          "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": scan_bytes / (scan_us * 1e-6) / 1e9 / HBM_PEAK_GBS,
                          "traffic": traffic_from_profiles(wl.name, "scan")},
    })
    if head is not None:
        # stage "expand" is the head path's tree kernel; no counter record is kept for it
        res["config"].update(d_H=w.d_e, rank=HEAD_RANK)
        res["roofline"]["kernel"] = "head_tree"
        res["roofline"]["traffic"] = None

    if args.copy_calibration:
        x = torch.empty(256 * 2**20 // 4, dtype=torch.float32, device=dev).fill_(1.0)
        y = torch.empty_like(x)
        y.copy_(x)
        torch.cuda.synchronize()

    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl.name, wl, bufs_host, args.cpu_seconds,
                                           SCORERS[args.scorer], head)
    plan.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

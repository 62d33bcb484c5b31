"""Tree parity: dt_build_tree (all of S1-S5 on the GPU) against the oracle.

Wherever the oracle's decisive score gaps exceed 1e-4 the trees must be
identical (tokens, parents, depth, position ids, mask, node count) and the
scores within 1e-4 (fp32 inputs) or 2e-2 (bf16 inputs feeding the
correction).  Seeds with smaller gaps must still give a valid best-first tree
within tolerance.  Sizes span several tiles and ragged tails; the full
Qwen3-shaped workloads are checked on sampled trees.
"""
import functools

import numpy as np
import pytest
import torch

import oracle
from gpu_util import DeviceWorkload, compare_tree
from paper_2607_08642_amd import binding, synth

pytestmark = pytest.mark.gpu


def run_case(wl, trees=None, name="", **kw):
    print(f"[tree] {name} batch={wl.batch} L={wl.L} M={wl.M} B={wl.B} T={wl.T} kw={kw}", flush=True)
    dw = DeviceWorkload(wl, **kw)
    try:
        got = dw.run()
    finally:
        dw.close()
    kinds = []
    for t in (range(wl.batch) if trees is None else trees):
        kinds.append(compare_tree(wl, t, got, dw.kw))
    print(f"[tree] {name}: {[k for k, _ in kinds]} max score err {max(e for _, e in kinds):.2e}",
          flush=True)
    return kinds, got


def test_tiny_workload():
    kinds, _ = run_case(synth.tiny(), name="tiny")
    assert kinds[0][0] == "exact"


SWEEP = [
    # (seed, batch, L, V, M, B, T, d_e, d_h, dtype, kw, extra)
    (1, 1, 4, 300, 8, 8, 0.0, 64, 32, synth.DT_F32, {}, {}),
    (2, 3, 6, 500, 16, 24, 0.7, 64, 64, synth.DT_F32, {}, dict(h0=True)),
    (3, 2, 5, 1000, 64, 16, 1.0, 128, 64, synth.DT_BF16, {}, {}),
    (4, 8, 3, 200, 12, 10, 1.5, 40, 32, synth.DT_F32, dict(max_children=3), dict(h0=True)),
    (5, 4, 8, 700, 32, 16, 0.0, 96, 64, synth.DT_BF16, dict(norm_mode=1), {}),
    (6, 1, 1, 100, 8, 6, 0.0, 32, 32, synth.DT_F32, {}, {}),
    (7, 5, 4, 400, 16, 1, 0.9, 32, 32, synth.DT_F32, {}, dict(h0=True)),
    (8, 2, 6, 300, 8, 6, 0.0, 64, 32, synth.DT_F32, dict(max_children=1), {}),
    (9, 3, 10, 2000, 64, 48, 0.8, 64, 64, synth.DT_BF16, dict(pos_offset=11), dict(h0=True)),
    (10, 2, 4, 64, 64, 20, 1.0, 32, 32, synth.DT_F32, {}, {}),
    (11, 1, 5, 333, 20, 30, 0.6, 36, 32, synth.DT_BF16, dict(max_children=8), {}),
    (12, 6, 16, 1500, 64, 64, 0.0, 64, 96, synth.DT_BF16, {}, dict(h0=True)),
    # several segment lists per row (10240 logits each): the register tree
    # merge with M < 64 and a 5-element last list, the one-wave merge of two
    # lists, more than 16 lists (block merge) and M > 64 (block merges)
    (13, 1, 4, 30725, 48, 16, 0.8, 32, 32, synth.DT_F32, {}, {}),
    (14, 2, 3, 15000, 40, 12, 0.0, 32, 32, synth.DT_BF16, {}, {}),
    (15, 1, 4, 200000, 32, 16, 1.0, 32, 32, synth.DT_F32, {}, {}),
    (16, 2, 4, 50000, 100, 24, 0.7, 32, 32, synth.DT_BF16, {}, dict(h0=True)),
    # the envelope's maxima: L = 64, M = 256, B = 256
    (17, 1, 64, 3000, 256, 256, 0.9, 32, 32, synth.DT_F32, {}, {}),
]


# the ablation arms (Appendix D): Marg (scorer 1) and Cond-static (scorer 2)
ARM_CASES = [c for c in SWEEP if c[0] in (2, 3, 5, 9, 12, 13, 14)]


@pytest.mark.parametrize("scorer", [1, 2], ids=["marg", "static"])
@pytest.mark.parametrize("case", ARM_CASES, ids=[f"s{c[0]}" for c in ARM_CASES])
def test_ablation_arms(case, scorer):
    seed, batch, L, V, M, B, T, d_e, d_h, dt, kw, extra = case
    wl = synth.random_small(seed, batch=batch, L=L, V=V, M=M, B=B, T=T, d_e=d_e, d_h=d_h,
                            dtype=dt, **extra)
    # (path-independent menus over bf16 logits tie exactly more often: a tree
    # with a tie is checked as a valid best-first tree within tolerance)
    run_case(wl, name=f"arm{scorer}-s{seed}", scorer=scorer, **kw)


@pytest.mark.parametrize("scorer", [1, 2], ids=["marg", "static"])
def test_ablation_arms_qwen_shape(scorer):
    wl = synth.WORKLOADS["qwen3_8b"]()
    kinds, _ = run_case(wl, name=f"arm{scorer}-qwen3_8b", scorer=scorer)
    # Marg's shared menus of bf16 logits hold exact ties here (checked as a valid
    # best-first tree within tolerance); the corrected menus of Cond-static do not
    assert kinds[0][0] == "exact" or scorer == 1


@pytest.mark.parametrize("case", SWEEP, ids=[f"s{c[0]}" for c in SWEEP])
def test_random_sweep(case):
    seed, batch, L, V, M, B, T, d_e, d_h, dt, kw, extra = case
    wl = synth.random_small(seed, batch=batch, L=L, V=V, M=M, B=B, T=T, d_e=d_e, d_h=d_h,
                            dtype=dt, **extra)
    kinds, _ = run_case(wl, name=f"sweep{seed}", **kw)
    assert sum(k == "exact" for k, _ in kinds) >= len(kinds) // 2


def test_greedy_chain_on_gpu():
    wl = synth.random_small(21, batch=2, L=6, V=400, M=16, B=6, T=0.0, d_e=64, d_h=32, h0=True)
    kinds, got = run_case(wl, name="chain", max_children=1)
    for t in range(2):
        np.testing.assert_array_equal(got["parents"][t], np.arange(-1, 5))


def test_zeroed_correction_on_gpu():
    wl = synth.random_small(22, batch=2, L=5, V=800, M=32, B=20, T=0.8, d_e=64, d_h=32)
    wl.weights.w_c = np.zeros_like(wl.weights.w_c)
    wl.weights.b_c = np.zeros_like(wl.weights.b_c)
    run_case(wl, name="zeroed")


def test_nonfinite_tree_isolated():
    wl = synth.random_small(23, batch=3, L=4, V=300, M=8, B=8, T=0.0, d_e=32, d_h=32)
    x = wl.logits.copy()
    x[1, 2, 5] = np.nan
    wl.logits = x
    kinds, got = run_case(wl, name="nan")
    assert got["status"][1] == binding.DT_TREE_NONFINITE and got["n_nodes"][1] == 0
    assert got["status"][0] == 0 and got["status"][2] == 0


def test_determinism_and_stream():
    wl = synth.random_small(24, batch=4, L=6, V=900, M=32, B=16, T=0.7, d_e=64, d_h=64,
                            dtype=synth.DT_BF16, h0=True)
    dw = DeviceWorkload(wl)
    try:
        a = dw.run()
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            b = dw.run()
    finally:
        dw.close()
    for k in a:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)


@functools.lru_cache(maxsize=None)
def qwen(name):
    return synth.WORKLOADS[name]()


@pytest.mark.parametrize("name", ["qwen3_4b", "qwen3_8b", "budget64"])
def test_qwen_workloads(name):
    run_case(qwen(name), name=name)


def test_qwen3_8b_paper_branching():
    run_case(qwen("qwen3_8b"), name="qwen3_8b-k8", max_children=8)


def test_concurrent_workload_sampled():
    run_case(qwen("concurrent"), trees=[0, 1, 7, 19, 31], name="concurrent")


def test_stage_timing_means():
    # profiling records every call's stage events; stage_ms gives their means
    wl = synth.random_small(31, batch=2, L=4, V=2000, M=16, B=8, T=0.5, d_e=32, d_h=64)
    dw = DeviceWorkload(wl)
    try:
        with pytest.raises(binding.DTError):
            dw.plan.stage_ms()                    # nothing profiled yet
        dw.plan.set_profiling(1)
        for _ in range(5):
            dw.run()
        ms = dw.plan.stage_ms()
        assert set(ms) == set(binding.STAGES)
        assert all(0.0 < v < 1000.0 for v in ms.values()), ms
        dw.plan.set_profiling(1)                  # a new count
        with pytest.raises(binding.DTError):
            dw.plan.stage_ms()
        dw.plan.set_profiling(0)
    finally:
        dw.close()


FIELDS = ("tokens", "parents", "depth", "position_ids", "mask", "scores", "n_nodes", "status")


def _snapshot(tree):
    return {k: getattr(tree, k).cpu().numpy().copy() for k in FIELDS}


def _assert_same(a, b, what):
    for k in FIELDS:
        np.testing.assert_array_equal(a[k], b[k], err_msg=f"{what}: {k}")


@pytest.mark.parametrize("name", ["qwen3_8b", "budget64"])
def test_repeatable_at_qwen_shape(name):
    # every reduction runs in a fixed order: repeated calls give identical bits
    wl = qwen(name)
    dw = DeviceWorkload(wl)
    try:
        first = dw.run()
        for rep in range(4):
            again = dw.run()
            for k in first:
                np.testing.assert_array_equal(first[k], again[k], err_msg=f"rep {rep}: {k}")
    finally:
        dw.close()


def test_graph_replay_matches_eager():
    # three calls on three logit buffers captured into one HIP graph; every
    # replay (with eager work and synchronisation in between) must reproduce
    # the eager trees bit for bit
    wl = qwen("qwen3_8b")
    dw = DeviceWorkload(wl)
    try:
        plan = dw.plan
        bufs = [dw.logits] + [torch.from_numpy(synth.logits_buffer(wl.name, i, wl.batch).view(np.int16))
                              .cuda().view(torch.bfloat16) for i in (1, 2)]
        outs = [binding.Tree.empty(wl.batch, wl.B, "cuda") for _ in bufs]
        ws = plan.workspace(wl.batch)
        for b, o in zip(bufs, outs):
            plan.build_tree(b, wl.T, dw.h0, out=o, workspace=ws)
        torch.cuda.synchronize()
        eager = [_snapshot(o) for o in outs]
        assert not all(np.array_equal(eager[0]["tokens"], e["tokens"]) for e in eager[1:])
        plan.set_profiling(1)            # capture records no events and counts no calls
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for b, o in zip(bufs, outs):
                plan.build_tree(b, wl.T, dw.h0, out=o, workspace=ws)
        with pytest.raises(binding.DTError):
            plan.stage_ms()
        plan.set_profiling(0)
        for rep in range(3):
            for o in outs:
                o.tokens.fill_(-5)
                o.scores.fill_(7.0)
                o.mask.fill_(3)
                o.n_nodes.fill_(-1)
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for i, o in enumerate(outs):
                _assert_same(_snapshot(o), eager[i], f"replay {rep} call {i}")
            plan.build_tree(bufs[rep], wl.T, dw.h0, out=outs[rep], workspace=ws)  # eager between
            torch.cuda.synchronize()
            _assert_same(_snapshot(outs[rep]), eager[rep], f"eager after replay {rep}")
        del g
    finally:
        dw.close()

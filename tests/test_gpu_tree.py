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
from helpers import run_oracle
from paper_2607_08642_amd import binding, synth

pytestmark = pytest.mark.gpu


# the kernels keep fp32 intermediates: at the Qwen3 shapes (bf16 inputs, whose
# contractual tolerance is 2e-2) the score error is held to the fp32 bar
QWEN_TOL = 1e-4


def run_case(wl, trees=None, name="", tol=None, **kw):
    print(f"[tree] {name} batch={wl.batch} L={wl.L} M={wl.M} B={wl.B} T={wl.T} kw={kw}", flush=True)
    dw = DeviceWorkload(wl, **kw)
    try:
        got = dw.run()
    finally:
        dw.close()
    kinds = []
    for t in (range(wl.batch) if trees is None else trees):
        kinds.append(compare_tree(wl, t, got, dw.kw, tol=tol, name=name))
    print(f"[tree] {name}: {[k for k, _ in kinds]} max score err {max(e for _, e in kinds):.2e}",
          flush=True)
    return kinds, got


def assert_identical(got, ref, t=0, what=""):
    n = ref["n_nodes"]
    assert int(got["n_nodes"][t]) == n, what
    for key in ("tokens", "parents", "depth", "position_ids", "mask"):
        np.testing.assert_array_equal(got[key][t], ref[key], err_msg=f"{what} {key}")


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
    assert any(k == "exact" for k, _ in kinds)


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


def _masked(seed, dtype):
    # vocabulary masks: rows whose finite logits number fewer than M (dead
    # candidate slots with id -1), a row with one finite logit, and rows with
    # fewer finite logits than B
    wl = synth.random_small(seed, batch=3, L=5, V=700, M=16, B=12, T=0.8, d_e=48, d_h=32,
                            dtype=dtype)
    x = synth.bf16_bits_to_f32(wl.logits) if dtype == synth.DT_BF16 else wl.logits.copy()
    rng = np.random.default_rng(seed)
    for t, r, n in ((0, 1, 5), (1, 0, 1), (1, 3, 6), (2, 2, 9), (2, 4, 3)):
        row = np.full(700, -np.inf, np.float32)
        idx = rng.choice(700, size=n, replace=False)
        row[idx] = x[t, r, idx]
        x[t, r] = row
    wl.logits = synth.f32_to_bf16_bits(x) if dtype == synth.DT_BF16 else x
    return wl


@pytest.mark.parametrize("dtype", [synth.DT_F32, synth.DT_BF16], ids=["f32", "bf16"])
def test_masked_rows(dtype):
    wl = _masked(31 + dtype, dtype)
    kinds, got = run_case(wl, name=f"masked {dtype}")
    assert all(int(s) == 0 for s in got["status"][: wl.batch])


@pytest.mark.parametrize("T", [0.1, 3.0])
def test_extreme_temperatures(T):
    # sharp and flat menus: exponent arguments far from the row maxima (the
    # scan's two exponent forms, the children's normalisation)
    wl = synth.random_small(41, batch=2, L=5, V=900, M=24, B=16, T=T, d_e=48, d_h=32,
                            dtype=synth.DT_BF16, h0=True)
    run_case(wl, name=f"T={T}")


def test_shifted_logits():
    # a constant added to every logit changes no log-probability: the tree of
    # logits offset by 3000 (fp32) is the oracle's tree of those logits
    wl = synth.random_small(43, batch=2, L=5, V=900, M=24, B=16, T=0.8, d_e=48, d_h=32, h0=True)
    wl.logits = (wl.logits + np.float32(3000.0)).astype(np.float32)
    run_case(wl, name="shifted")


@pytest.mark.parametrize("L,M,B", [(2, 4, 30), (1, 5, 12), (3, 3, 64)])
def test_budget_beyond_reachable_nodes(L, M, B):
    # every node the depth limit and the menus allow (M + M^2 + ... < B) is in
    # the tree, which ends short of B
    wl = synth.random_small(51, batch=2, L=L, V=200, M=M, B=B, T=0.9, d_e=32, d_h=32)
    kinds, got = run_case(wl, name=f"short L={L} M={M} B={B}")
    reach = sum(M ** d for d in range(1, L + 1))
    assert all(int(n) == reach for n in got["n_nodes"][: wl.batch])


@pytest.mark.parametrize("batch,d_h", [(100, 64), (300, 32)])
def test_many_trees_per_call(batch, d_h):
    # more trees than XCD classes hold at once: 100 trees of two members each
    # (13 per class, start-order member slots) and 300 one-member trees (more
    # workgroups than CUs)
    wl = synth.random_small(81, batch=batch, L=4, V=300, M=8, B=10, T=0.8, d_e=32, d_h=d_h,
                            h0=True)
    run_case(wl, name=f"batch {batch}")


@pytest.mark.parametrize("d_h,batch", [(160, 2), (768, 1), (1024, 1), (1024, 9)])
def test_state_widths(d_h, batch):
    # path-state widths off the tested grid: 160 (two members of 80 units), 768
    # and 1024 (the largest), whose sixteen-member layouts exceed the LDS: eight
    # members of 96 and 128 units
    wl = synth.random_small(91, batch=batch, L=5, V=600, M=16, B=14, T=0.8, d_e=64, d_h=d_h,
                            h0=True, w_scale=0.2)
    run_case(wl, name=f"d_h {d_h} batch {batch}")


def test_single_candidate_rows():
    # M = 1: every menu holds one token, so the tree is the chain of the rows' top
    # tokens (min(B, L) nodes)
    wl = synth.random_small(92, batch=2, L=7, V=500, M=1, B=5, T=0.8, d_e=32, d_h=32)
    kinds, got = run_case(wl, name="M=1")
    for t in range(2):
        np.testing.assert_array_equal(got["parents"][t][:5], np.arange(-1, 4))


def test_menus_of_the_whole_vocabulary():
    # M = V: every token is a candidate, the tail is empty (R = -inf)
    for norm_mode in (0, 1):
        wl = synth.random_small(93, batch=2, L=4, V=64, M=64, B=20, T=0.9, d_e=32, d_h=32)
        run_case(wl, name=f"M=V norm {norm_mode}", norm_mode=norm_mode)


def test_odd_vocabulary_at_qwen_width():
    # a vocabulary of 151937 bf16 logits (rows not 16-byte aligned: the block
    # scan kernel, fifteen segment lists per row) at d_h = 512, M = 64
    wl = synth.random_small(94, batch=1, L=4, V=151937, M=64, B=16, T=1.0, d_e=64, d_h=512,
                            dtype=synth.DT_BF16, w_scale=0.1)
    run_case(wl, name="odd V")


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
    kinds, _ = run_case(qwen(name), name=name, tol=QWEN_TOL)
    if name != "qwen3_8b":                 # (qwen3_8b holds a 5.6e-5 near-tie: banded)
        assert kinds[0][0] == "exact"


def test_qwen3_8b_paper_branching():
    run_case(qwen("qwen3_8b"), name="qwen3_8b-k8", tol=QWEN_TOL, max_children=8)


def test_concurrent_workload_sampled():
    run_case(qwen("concurrent"), trees=[0, 1, 7, 19, 31], name="concurrent", tol=QWEN_TOL)


# ---- deep trees on the production instances (d_h = 512, M = 64, L = 16, bf16) ----
# one tree per call runs the 16-member instance, 32 trees the 8-member one

@pytest.mark.parametrize("k", [0, 8, 2, 1])
def test_deep_tree_at_qwen_shape(k):
    wl = qwen("deep")
    kinds, got = run_case(wl, name=f"deep-k{k}", tol=QWEN_TOL, max_children=k)
    assert kinds[0][0] == "exact"
    depth = int(got["depth"][0].max())
    assert depth >= (16 if k == 1 else 9), depth


def test_expand_stats_count_the_chain():
    # k = 1 over L = 16 is a chain: the root step plus one step per node above
    # depth L, each expanding exactly one node (the statistics the bench reads)
    wl = qwen("deep")
    dw = DeviceWorkload(wl, max_children=1)
    try:
        with pytest.raises(binding.DTError):
            dw.plan.expand_stats(1)             # nothing profiled yet
        dw.plan.set_profiling(1)
        got = dw.run()
        steps, expanded = dw.plan.expand_stats(1)
        dw.plan.set_profiling(0)
    finally:
        dw.close()
    assert int(got["depth"][0].max()) == 16
    assert steps == [16] and expanded == [16], (steps, expanded)


def test_deep_concurrent_all_trees():
    wl = qwen("deep_concurrent")
    kinds, got = run_case(wl, name="deep_concurrent", tol=QWEN_TOL)
    assert sum(k == "exact" for k, _ in kinds) >= 16
    assert int(got["depth"].max()) >= 12


def test_deep_qwen_shape_100_trees_sampled():
    # 100 deep Qwen3-8B-shaped trees in one call: two members per tree on the
    # generic instance (d_h 512 split in halves), 13 trees per XCD class
    wl = synth.deep_concurrent(batch=100)
    kinds, got = run_case(wl, trees=[0, 1, 49, 98, 99], name="deep x100", tol=QWEN_TOL)
    assert all(int(s) == 0 for s in got["status"][:100])


def test_twin_ties_at_qwen_shape():
    # every near-tie of this tree is an exact structural tie (twin tokens): the
    # GPU must order them by the heap's insertion order, node for node
    wl = synth.twin_tokens(qwen("deep"))
    for k in (0, 8):
        ref = run_oracle(wl, 0, max_children=k)
        assert all(v == 0.0 or v > 1e-4 for _, v in ref["gaps"])
        assert sum(v == 0.0 for _, v in ref["gaps"]) >= 8
        dw = DeviceWorkload(wl, max_children=k)
        try:
            got = dw.run()
        finally:
            dw.close()
        assert_identical(got, ref, what=f"twins k={k}")
        err = float(np.max(np.abs(got["scores"][0][:ref["n_nodes"]] - ref["scores"][:ref["n_nodes"]])))
        assert err <= QWEN_TOL, err
        print(f"[tree] twins k={k}: identical, score err {err:.2e}", flush=True)


# ---- exact ties at small shapes ----

def _tie_weights(V, d_e, d_h, rng=None, emb=None):
    z = lambda *s: np.zeros(s, np.float32)
    if rng is None:
        return synth.Weights(z(V, d_e), z(3 * d_h, d_e), z(3 * d_h, d_h), None, None, z(d_e, d_h),
                             z(d_e), synth.DT_F32, V, d_e, d_h)
    u = lambda *s: rng.uniform(-0.5, 0.5, s).astype(np.float32)
    return synth.Weights(emb, u(3 * d_h, d_e), u(3 * d_h, d_h), u(3 * d_h), u(3 * d_h), u(d_e, d_h),
                         u(d_e), synth.DT_F32, V, d_e, d_h)


def test_tie_rules_on_gpu():
    # the two hand-derived tie trees (tests/golden/tie_trees.json) at a width the
    # kernels take: zero correction with sibling and cross-parent ties, and twin
    # tokens under a nonzero GRU and head
    X = np.log(np.array([[0.3, 0.3, 0.2, 0.2], [0.25] * 4])).astype(np.float32)
    wl = synth.Workload("ties", X[None], synth.DT_F32, None, _tie_weights(4, 8, 32), 2, 4, 10,
                        0.0, 1)
    dw = DeviceWorkload(wl)
    try:
        got = dw.run()
    finally:
        dw.close()
    np.testing.assert_array_equal(got["tokens"][0], [0, 1, 2, 3, 0, 1, 2, 3, 0, 1])
    np.testing.assert_array_equal(got["parents"][0], [-1, -1, -1, -1, 0, 0, 0, 0, 1, 1])
    assert_identical(got, run_oracle(wl), what="sibling ties")
    rng = np.random.default_rng(5)
    emb = np.repeat(rng.uniform(-1, 1, (1, 8)).astype(np.float32), 2, axis=0)
    X = np.zeros((2, 2), np.float32)
    wl = synth.Workload("twins", X[None], synth.DT_F32, rng.uniform(-0.5, 0.5, (1, 32)).astype(np.float32),
                        _tie_weights(2, 8, 32, rng, emb), 2, 2, 5, 0.0, 1)
    dw = DeviceWorkload(wl)
    try:
        got = dw.run()
    finally:
        dw.close()
    np.testing.assert_array_equal(got["tokens"][0], [0, 1, 0, 1, 0])
    np.testing.assert_array_equal(got["parents"][0], [-1, -1, 0, 0, 1])
    assert_identical(got, run_oracle(wl), what="twin tokens")


def test_table_overflow_with_exact_ties():
    # Constant rows and zero correction: every child ties with its siblings and
    # cousins, B = 256 and k = M = 64, so one chunk of 16 depth-1 nodes appends
    # 1,024 tied children; every node stays a candidate (all score >= vB), the
    # candidate list outgrows its score buffer and the next chunk overflows the
    # node table (the table's ranking path).  The tree is flagged truncated; its
    # first 256 pops (64 depth-1 nodes, then the children of the first three by
    # insertion order) were appended before the overflow and match the oracle's.
    V, L, M, B = 128, 4, 64, 256
    X = np.zeros((L, V), np.float32)
    wl = synth.Workload("overflow", X[None], synth.DT_F32, None, _tie_weights(V, 8, 32), L, M, B, 0.0, 1)
    ref = run_oracle(wl)
    dw = DeviceWorkload(wl)
    try:
        got = dw.run()
    finally:
        dw.close()
    assert int(got["status"][0]) & binding.DT_TREE_TRUNCATED, got["status"][0]
    n = int(got["n_nodes"][0])
    assert n == ref["n_nodes"] == B, (n, ref["n_nodes"])
    for key in ("tokens", "parents", "depth", "position_ids"):
        np.testing.assert_array_equal(got[key][0][:n], ref[key][:n], err_msg=key)
    np.testing.assert_allclose(got["scores"][0][:n], ref["scores"][:n], rtol=0, atol=1e-5)
    print(f"[tree] table overflow: truncated, {n} pops identical", flush=True)


def test_marg_integer_logit_ties_on_gpu():
    # Marg over rows with repeated logit values: siblings tie exactly (slot order
    # decides) and so do their children across parents (insertion order decides);
    # the values are chosen so that no other near-tie exists
    rng = np.random.default_rng(9)
    V, M, B = 300, 16, 40
    X = (rng.standard_normal((2, V)) * 0.3 - 3.0).astype(np.float32)
    X[0, rng.choice(V, 4, replace=False)] = 5.0
    X[0, rng.choice(V, 6, replace=False)] = 2.0
    X[1, rng.choice(V, 3, replace=False)] = 4.0
    X[1, rng.choice(V, 5, replace=False)] = 1.5
    w = synth.random_small(33, batch=1, L=2, V=V, M=M, B=B, T=0.0, d_e=16, d_h=32).weights
    wl = synth.Workload("marg_ties", X[None], synth.DT_F32, None, w, 2, M, B, 0.0, 1)
    ref = run_oracle(wl, 0, scorer=oracle.SCORER_MARG)
    assert all(v == 0.0 or v > 1e-4 for _, v in ref["gaps"])
    assert sum(v == 0.0 for _, v in ref["gaps"]) >= 10
    dw = DeviceWorkload(wl, scorer=oracle.SCORER_MARG)
    try:
        got = dw.run()
    finally:
        dw.close()
    assert_identical(got, ref, what="marg ties")


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


def test_repeatable_under_concurrent_load():
    # 32 trees per call (every scan wave streaming several batches): the same
    # bits whether the calls run alone or beside heavy copies on another stream,
    # which shifts the waves' relative timing -- the scan's bounds, candidates
    # and tail sums must not depend on it
    wl = qwen("concurrent")
    dw = DeviceWorkload(wl)
    src = torch.empty(2**28 // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    side = torch.cuda.Stream()
    try:
        first = dw.run()
        for rep in range(3):
            with torch.cuda.stream(side):
                for _ in range(4):
                    dst.copy_(src)
            again = dw.run()
            side.synchronize()
            for k in first:
                np.testing.assert_array_equal(first[k], again[k], err_msg=f"rep {rep}: {k}")
        ids, vals, tail, flags = binding.scan_topm(dw.logits.view(-1, wl.weights.V), wl.M, wl.T)
        torch.cuda.synchronize()
        t0 = tail.cpu().numpy()
        for rep in range(3):
            with torch.cuda.stream(side):
                for _ in range(4):
                    dst.copy_(src)
            _, _, tail2, _ = binding.scan_topm(dw.logits.view(-1, wl.weights.V), wl.M, wl.T)
            side.synchronize()
            np.testing.assert_array_equal(t0, tail2.cpu().numpy(), err_msg=f"scan rep {rep}")
    finally:
        dw.close()

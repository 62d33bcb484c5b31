"""The frontier builder on the GPU (dt_options.frontier_width; Appendix B's
ledger and selection) against the oracle's, through the C ABI, at W = 1, 4
and B on small cases, the three scorers and the Qwen3-8B-shaped deep trees on
both production instances.  At W = B the tree must also be the heap's.
"""
import numpy as np
import pytest

import oracle
from gpu_util import DeviceWorkload, compare_tree
from helpers import run_oracle
from paper_2607_08642_amd import binding, synth

pytestmark = pytest.mark.gpu
QWEN_TOL = 1e-4


def run_frontier(wl, W, name, trees=None, tol=None, **kw):
    print(f"[frontier] {name} W={W} batch={wl.batch} L={wl.L} M={wl.M} B={wl.B} kw={kw}",
          flush=True)
    dw = DeviceWorkload(wl, frontier_width=W, **kw)
    try:
        got = dw.run()
    finally:
        dw.close()
    kinds = [compare_tree(wl, t, got, dict(dw.kw), tol=tol, name=f"frontier-{name}-W{W}")
             for t in (range(wl.batch) if trees is None else trees)]
    print(f"[frontier] {name} W={W}: {[k for k, _ in kinds]} "
          f"max err {max(e for _, e in kinds):.2e}", flush=True)
    return kinds, got


CASES = [
    # (seed, batch, L, V, M, B, T, d_e, d_h, dtype, kw, extra)
    (2, 3, 6, 500, 16, 24, 0.7, 64, 64, synth.DT_F32, {}, dict(h0=True)),
    (5, 4, 8, 700, 32, 16, 0.0, 96, 64, synth.DT_BF16, dict(norm_mode=1), {}),
    (9, 3, 10, 2000, 64, 48, 0.8, 64, 64, synth.DT_BF16, dict(max_children=8), dict(h0=True)),
    (12, 6, 16, 1500, 64, 64, 0.0, 64, 96, synth.DT_BF16, {}, dict(h0=True)),
]


@pytest.mark.parametrize("W", [1, 4, "B"])
@pytest.mark.parametrize("case", CASES, ids=[f"s{c[0]}" for c in CASES])
def test_frontier_small(case, W):
    seed, batch, L, V, M, B, T, d_e, d_h, dt, kw, extra = case
    wl = synth.random_small(seed, batch=batch, L=L, V=V, M=M, B=B, T=T, d_e=d_e, d_h=d_h,
                            dtype=dt, **extra)
    W = B if W == "B" else W
    kinds, got = run_frontier(wl, W, f"s{seed}", **kw)
    assert any(k == "exact" for k, _ in kinds)
    if W == B:
        # the heap's tree, wherever its decisive gaps leave no choice
        for t in range(batch):
            ref = run_oracle(wl, t, **kw)
            if ref["min_gap"] > 1e-4:
                for key in ("tokens", "parents", "depth", "mask"):
                    np.testing.assert_array_equal(got[key][t], ref[key], err_msg=f"{t} {key}")


@pytest.mark.parametrize("W", [1, 3])
def test_frontier_masked_rows_and_short_budget(W):
    # vocabulary-masked rows (fewer finite logits than M, one row with a
    # single finite logit), and a budget the frontier cannot fill (L = 2, M = 4)
    wl = synth.random_small(71, batch=2, L=5, V=600, M=16, B=12, T=0.8, d_e=48, d_h=32)
    x = wl.logits.copy()
    rng = np.random.default_rng(71)
    for t, r, n in ((0, 1, 5), (1, 0, 1), (1, 2, 4)):
        row = np.full(600, -np.inf, np.float32)
        idx = rng.choice(600, size=n, replace=False)
        row[idx] = x[t, r, idx]
        x[t, r] = row
    wl.logits = x
    run_frontier(wl, W, "masked")
    wl = synth.random_small(72, batch=2, L=2, V=200, M=4, B=30, T=0.9, d_e=32, d_h=32)
    kinds, got = run_frontier(wl, W, "short")
    for t in range(wl.batch):
        assert int(got["n_nodes"][t]) == run_oracle(wl, t, frontier_width=W)["n_nodes"] < 30


@pytest.mark.parametrize("scorer", [1, 2], ids=["marg", "static"])
def test_frontier_ablation_arms(scorer):
    wl = synth.random_small(2, batch=3, L=6, V=500, M=16, B=24, T=0.7, d_e=64, d_h=64, h0=True)
    run_frontier(wl, 4, f"arm{scorer}", scorer=scorer)


@pytest.mark.parametrize("W", [1, 4, 16])
def test_frontier_deep_qwen_shape(W):
    # one tree per call: the 16-member production instance
    kinds, got = run_frontier(synth.deep(), W, "deep", tol=QWEN_TOL)
    assert kinds[0][0] == "exact"


def test_frontier_deep_concurrent_sampled():
    # 32 trees per call: the 8-member production instance
    kinds, _ = run_frontier(synth.deep_concurrent(), 4, "deep_concurrent", trees=[0, 5, 13, 22, 31],
                            tol=QWEN_TOL)
    assert sum(k == "exact" for k, _ in kinds) >= 3


def test_frontier_rejects_head_and_adaptive_budget():
    wl = synth.random_small(3, batch=1, L=4, V=300, M=16, B=8, T=0.0, d_e=32, d_h=32)
    dw = DeviceWorkload(wl, frontier_width=2)
    try:
        with pytest.raises(binding.DTError) as e:
            dw.plan.set_adaptive_budget(1.0, [0.0] * (wl.B + 1))
        assert e.value.status == -4
    finally:
        dw.close()

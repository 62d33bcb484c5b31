"""Pins of the oracle's frontier builder (Appendix B, frontier ledger and
selection; the batched construction for serving, section 4.5.1; CPU only).

* W >= B selects the heap's tree: identical arrays on tie-free inputs (the
  equivalence argument of Appendix B), for several k, h0, T and both
  normalisations;
* a hand-derived W = 1 tree on the factorised golden rows, which differs from
  the heap's (the second depth-1 lane is evicted before its child is scored);
* W = 1, 2, 3 against the independent full-vocabulary frontier builder in
  tests/indep.py (node sets on tie-free inputs);
* the frontier cut's gap (W-th vs (W+1)-th score of a depth) is logged.
"""
import numpy as np
import pytest

import indep
import oracle
from helpers import run_oracle
from paper_2607_08642_amd import synth

FIELDS = ("tokens", "parents", "depth", "position_ids", "mask", "n_nodes")


def small(seed, **kw):
    args = dict(batch=1, L=4, V=40, M=6, B=10, T=0.8, d_e=6, d_h=5, emb_std=0.8, w_scale=0.8,
                logit_scale=1.0, spikes=1, spike=1.0, h0=True)
    args.update(kw)
    return synth.random_small(seed, **args)


@pytest.mark.parametrize("seed", range(6))
def test_width_at_least_budget_is_heap_tree(seed):
    kw = [dict(), dict(max_children=3), dict(norm_mode=oracle.NORM_SLICE), dict(max_children=1),
          dict(pos_offset=5), dict(max_children=2)][seed]
    wl = small(900 + seed, T=[0.0, 0.7, 1.3][seed % 3], h0=bool(seed % 2))
    heap = run_oracle(wl, **kw)
    assert heap["min_gap"] > 1e-9
    for W in (wl.B, wl.B + 7):
        fr = run_oracle(wl, frontier_width=W, **kw)
        for k in FIELDS:
            np.testing.assert_array_equal(fr[k], heap[k], err_msg=f"W={W} {k}")
        np.testing.assert_allclose(fr["scores"], heap["scores"], atol=1e-12)


def test_hand_derived_width_one():
    # rows log(.5 .25 .125 .125), log(.1 .6 .2 .1), M = k = 2, zero correction, B = 4.
    # Depth 1 ledger: (0) .5, (1) .25; W = 1 keeps lane (0).  Depth 2 ledger:
    # (0,1) .3, (0,2) .1 (the children of (1) are never scored).  Global top 4 by
    # g: (0) .5, (0,1) .3, (1) .25, (0,2) .1 -- the heap would take (1,1) .15 last.
    X = np.log(np.array([[0.5, 0.25, 0.125, 0.125], [0.1, 0.6, 0.2, 0.1]])).astype(np.float32)
    z = np.zeros
    w = dict(w_ih=z((3, 1), np.float32), w_hh=z((3, 1), np.float32), b_ih=None, b_hh=None,
             w_c=z((1, 1), np.float32), b_c=z(1, np.float32), dtype=oracle.DT_F32)
    emb = z((4, 1), np.float32)
    fr = oracle.build_tree(X, emb, oracle.DT_F32, w, None, 2, 4, 0.0, frontier_width=1)
    assert fr["tokens"][:4].tolist() == [0, 1, 1, 2]
    assert fr["parents"][:4].tolist() == [-1, 0, -1, 0]
    assert fr["depth"][:4].tolist() == [1, 2, 1, 2]
    np.testing.assert_allclose(np.exp(fr["scores"][:4]), [0.5, 0.3, 0.25, 0.1], atol=1e-6)
    assert fr["mask"][:4, :4].tolist() == [[1, 0, 0, 0], [1, 1, 0, 0], [0, 0, 1, 0], [1, 0, 0, 1]]
    heap = oracle.build_tree(X, emb, oracle.DT_F32, w, None, 2, 4, 0.0)
    assert heap["tokens"][:4].tolist() == [0, 1, 1, 1]        # (1,1) .15 instead
    # the frontier cut at depth 1: ln(.5) - ln(.25)
    assert [v for k, v in fr["gaps"] if k == "frontier"] == pytest.approx([np.log(2.0)], abs=1e-6)


@pytest.mark.parametrize("W", [1, 2, 3])
@pytest.mark.parametrize("seed", range(3))
def test_narrow_frontier_against_independent_builder(seed, W):
    wl = small(950 + seed, L=4, V=12, M=5, B=8)
    k = min(wl.M, wl.B)
    fr = run_oracle(wl, frontier_width=W)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, wl.h0[0], wl.M, wl.T)
    want = indep.frontier_tree(sc, wl.B, k, W)
    got = set(indep.tree_paths(fr["tokens"], fr["parents"], fr["n_nodes"]))
    assert got == want
    # parents first, scores non-increasing in the emitted order
    s = fr["scores"][:fr["n_nodes"]]
    assert np.all(s[1:] <= s[:-1])
    assert all(fr["parents"][i] < i for i in range(fr["n_nodes"]))


def test_narrow_frontier_differs_from_heap_somewhere():
    # W < B is an approximation: on these seeds at least one tree differs
    diffs = 0
    for seed in range(6):
        wl = small(970 + seed, L=5, V=20, M=6, B=12)
        heap = run_oracle(wl)
        fr = run_oracle(wl, frontier_width=2)
        diffs += not np.array_equal(heap["tokens"], fr["tokens"])
    assert diffs >= 1

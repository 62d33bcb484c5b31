"""Pins of the oracle's tie rules, decisive-gap log and re-scorer (CPU only).

* Hand-derived trees with exact ties (tests/golden/tie_trees.json): children
  of an expansion in (log-prob desc, slot asc) order, equal heap scores popped
  in insertion order (Appendix B; Alg. 1 steps 3-4).  Reversing either rule
  is a planted mistake that these trees catch.
* Hand-derived decisive gaps (tests/golden/gap_cases.json): each of the three
  gap kinds is the smallest in one case, with the best excluded heap score.
* score_paths: reproduces the cumulative log-prob of every path of the
  k-restricted candidate tree as enumerated by the independent full-vocabulary
  scorer, rejects a child outside the top k, and accepts it under a tie
  tolerance exactly when its log-prob is that close to the k-th.
"""
import heapq as hq
import json
import math
import os

import numpy as np
import pytest

import indep
import oracle
import oracle.dominotree_ref as ref
from helpers import rescore, run_oracle
from paper_2607_08642_amd import synth

HERE = os.path.dirname(__file__)
TIES = os.path.join(HERE, "golden", "tie_trees.json")
GAPS = os.path.join(HERE, "golden", "gap_cases.json")


def _case_inputs(c):
    X = np.log(np.array(c["logits_probs"], np.float64)).astype(np.float32)
    z1 = [[0.0]] * 3
    w = dict(w_ih=np.array(c.get("w_ih", z1), np.float32), w_hh=np.array(c.get("w_hh", z1), np.float32),
             b_ih=None, b_hh=None, w_c=np.array(c.get("w_c", [[0.0]]), np.float32),
             b_c=np.array(c.get("b_c", [0.0]), np.float32), dtype=oracle.DT_F32)
    emb = np.array(c.get("emb", [[0.0]] * c["V"]), np.float32)
    h0 = np.array(c.get("h0", [0.0] * w["w_hh"].shape[1]), np.float64)
    return X, emb, w, h0


def _run_case(c):
    X, emb, w, h0 = _case_inputs(c)
    return oracle.build_tree(X, emb, oracle.DT_F32, w, h0, c["M"], c["B"], c.get("T", 0.0),
                             max_children=c.get("max_children", 0))


def tie_mismatch():
    for c in json.load(open(TIES))["cases"]:
        out, e = _run_case(c), c["expect"]
        n = len(e["tokens"])
        if out["n_nodes"] != n:
            return c["name"] + ": n_nodes"
        for key in ("tokens", "parents", "depth"):
            if out[key][:n].tolist() != e[key]:
                return f"{c['name']}: {key} {out[key][:n].tolist()}"
        if out["mask"][:n, :n].tolist() != e["mask"]:
            return c["name"] + ": mask"
        if np.max(np.abs(out["scores"][:n] - np.log(e["scores_probs"]))) > 1e-6:
            return c["name"] + ": scores"
    return None


def test_tie_golden_trees():
    assert tie_mismatch() is None


def test_tie_golden_ties_are_exact():
    # the equal scores of the hand cases are bit-identical in the oracle (gap 0.0)
    for c in json.load(open(TIES))["cases"]:
        out = _run_case(c)
        assert any(v == 0.0 for kind, v in out["gaps"] if kind == "pop"), c["name"]


def test_children_tie_rule_mistake_is_caught(monkeypatch):
    # (log-prob desc, slot DESC) instead of slot asc
    orig = ref._Model.children

    def bad(self, S, d, k, gaps):
        kids, ell_out = orig(self, S, d, k, gaps)
        return sorted(kids, key=lambda c: (-c[1], -c[2])), ell_out

    monkeypatch.setattr(ref._Model, "children", bad)
    assert tie_mismatch() is not None


def test_heap_tie_rule_mistake_is_caught(monkeypatch):
    # equal scores popped in REVERSE insertion order
    class LatestFirst:
        @staticmethod
        def heappush(h, e):
            hq.heappush(h, (e[0], -e[1]) + e[2:])

        @staticmethod
        def heappop(h):
            e = hq.heappop(h)
            return (e[0], -e[1]) + e[2:]

    monkeypatch.setattr(ref, "heapq", LatestFirst)
    assert tie_mismatch() is not None


@pytest.mark.parametrize("case", json.load(open(GAPS))["cases"], ids=lambda c: c["name"])
def test_gap_golden(case):
    out = _run_case(case)
    e = case["expect"]
    for kind in ("pop", "boundary", "children"):
        got = sorted(v for k, v in out["gaps"] if k == kind)
        want = sorted(math.log(a / b) for a, b in e[kind])
        assert len(got) == len(want), (kind, got, want)
        np.testing.assert_allclose(got, want, atol=1e-6, err_msg=kind)
    kind_min, v_min = min(out["gaps"], key=lambda kv: kv[1])
    assert kind_min == e["min_kind"]
    assert out["min_gap"] == v_min
    assert out["excluded"] == pytest.approx(math.log(e["excluded_prob"]), abs=1e-6)


def test_gap_log_matches_tree():
    # on a random tree: pop gaps are the consecutive score differences, the
    # boundary gap uses the best excluded score, min_gap is the minimum of all
    wl = synth.random_small(31, batch=1, L=4, V=40, M=6, B=9, T=0.8, d_e=6, d_h=5, h0=True)
    out = run_oracle(wl, max_children=3)
    n = out["n_nodes"]
    pops = [v for k, v in out["gaps"] if k == "pop"]
    np.testing.assert_array_equal(pops, out["scores"][:n - 1] - out["scores"][1:n])
    bnd = [v for k, v in out["gaps"] if k == "boundary"]
    assert bnd == [out["scores"][n - 1] - out["excluded"]]
    assert out["min_gap"] == min(v for _, v in out["gaps"])
    # per-node diagnostics: own log-prob, best slot cut off below it, sibling rank
    for i in range(n):
        p = out["parents"][i]
        gp = 0.0 if p < 0 else out["scores"][p]
        assert out["scores"][i] == pytest.approx(gp + out["ell"][i], abs=1e-12)
        assert out["ell_out"][i] <= out["ell"][i]
        assert 0 <= out["rank"][i] < 3


# ---------------------------------------------------------------------------
# score_paths against the independent brute-force enumeration
# ---------------------------------------------------------------------------

def _small(seed, **kw):
    args = dict(batch=1, L=3, V=12, M=5, B=6, T=0.7, d_e=6, d_h=5, emb_std=0.8, w_scale=0.8,
                logit_scale=1.0, spikes=1, spike=1.0, h0=True)
    args.update(kw)
    return synth.random_small(seed, **args)


def _chain(path):
    return list(path), list(range(-1, len(path) - 1))


@pytest.mark.parametrize("seed", range(3))
def test_score_paths_reproduces_brute_force(seed):
    wl = _small(50 + seed, T=[0.0, 0.7, 1.3][seed])
    k = 3
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, wl.h0[0], wl.M, wl.T)
    allp = indep.enumerate_paths(sc, k)
    for path, g in allp.items():
        toks, pars = _chain(path)
        gs, valid = rescore(wl, 0, toks, pars, len(toks), max_children=k)
        assert valid, path
        assert gs[-1] == pytest.approx(g, abs=1e-10), path
    # and on a whole tree (nodes in pop order, shared prefixes)
    out = run_oracle(wl, max_children=k)
    n = out["n_nodes"]
    gs, valid = rescore(wl, 0, out["tokens"], out["parents"], n, max_children=k)
    assert valid
    np.testing.assert_allclose(gs, out["scores"][:n], atol=1e-12)


def test_score_paths_rejects_non_top_k_child_and_tie_tolerance():
    wl = _small(60, L=2, M=6)
    k = 2
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, wl.h0[0], wl.M, wl.T)
    ranked = sc.ranked_children(sc.h0, 1, wl.M)          # every live slot of depth 1, in rank order
    assert len(ranked) > k
    (tk, lk), (tk1, lk1) = ranked[k - 1], ranked[k]      # the k-th and the (k+1)-th child
    gap = lk - lk1
    assert gap > 1e-6
    g, valid = rescore(wl, 0, [tk1], [-1], 1, max_children=k)
    assert not valid                                     # outside the top k
    g, valid = rescore(wl, 0, [tk1], [-1], 1, max_children=k, tie_tol=0.5 * gap)
    assert not valid                                     # still too far below the k-th
    g, valid = rescore(wl, 0, [tk1], [-1], 1, max_children=k, tie_tol=1.01 * gap)
    assert valid and g[0] == pytest.approx(lk1, abs=1e-10)
    # the (k+1)-th child's own child is scored along the (k+1)-th child's state
    S1 = sc.step(sc.h0, tk1)
    t2, l2 = sc.ranked_children(S1, 2, k)[0]
    g, valid = rescore(wl, 0, [tk1, t2], [-1, 0], 2, max_children=k, tie_tol=1.01 * gap)
    assert valid and g[1] == pytest.approx(lk1 + l2, abs=1e-10)


def test_score_paths_rejects_malformed_trees():
    wl = _small(61, L=2)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, wl.h0[0], wl.M, wl.T)
    t1 = sc.ranked_children(sc.h0, 1, 1)[0][0]
    t2 = sc.ranked_children(sc.step(sc.h0, t1), 2, 1)[0][0]
    assert rescore(wl, 0, [t1, t2], [-1, 0], 2)[1]
    assert not rescore(wl, 0, [t1, t2], [-1, 1], 2)[1]           # parent not earlier
    assert not rescore(wl, 0, [t1, t2, t2], [-1, 0, 1], 3)[1]    # below depth L
    outside = [v for v in range(wl.weights.V) if v not in sc.slices[0]][0]
    assert not rescore(wl, 0, [outside], [-1], 1)[1]             # not in the depth's slice

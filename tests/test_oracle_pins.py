"""Pins of the oracle against what the paper and the mathematics fix.

* brute force: the tree is the prefix-closed top-B set of the candidate tree by
  cumulative conditional log-prob (best-first over a monotone score, Appendix B);
* zeroed correction: the factorised top-B-by-product-of-marginals tree (DDTree's
  marginal heap, sections 2.4 and 3.1);
* B=1 / k=1: the greedy Domino chain (Fact A);
* a path-independent correction: a closed form over shifted marginals;
* frontier builder with W = B returns the same node set (Appendix B);
* invariants, temperature and M = V readings;
* hand-derived golden trees;
* planted mistakes in the oracle are caught by these pins.
"""
import json
import math
import os

import numpy as np
import pytest

import indep
import oracle
import oracle.dominotree_ref as ref
from helpers import check_tree_valid, run_oracle
from paper_2607_08642_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_trees.json")


def small(seed, **kw):
    args = dict(batch=1, L=3, V=10, M=4, B=6, T=0.0, d_e=6, d_h=5, emb_std=0.8,
                w_scale=0.8, logit_scale=1.0, spikes=1, spike=1.0)
    args.update(kw)
    return synth.random_small(seed, **args)


def oracle_paths(out):
    return indep.tree_paths(out["tokens"], out["parents"], out["n_nodes"])


def bruteforce_mismatch(wl, max_children=0, norm_slice=False):
    """None if the oracle tree equals the brute-force top-B set, else a message."""
    out = run_oracle(wl, max_children=max_children,
                     norm_mode=oracle.NORM_SLICE if norm_slice else oracle.NORM_TAIL)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights,
                           None if wl.h0 is None else wl.h0[0], wl.M, wl.T, norm_slice)
    k = min(wl.M, wl.B) if max_children <= 0 else min(max_children, wl.M)
    allp = indep.enumerate_paths(sc, k)
    top, gap = indep.top_b_paths(allp, wl.B)
    assert gap > 1e-9, "seed has ties at the budget boundary"
    got = oracle_paths(out)
    if set(got) != top:
        return f"node sets differ: {sorted(set(got) ^ top)}"
    for p, g in zip(got, out["scores"][: out["n_nodes"]]):
        if abs(allp[p] - g) > 1e-10:
            return f"score of {p}: {g} vs {allp[p]}"
    # prefix closure of the brute-force set
    for p in top:
        if len(p) > 1 and p[:-1] not in top:
            return "brute-force top-B not prefix-closed"
    return None


@pytest.mark.parametrize("seed", range(8))
def test_bruteforce_top_b(seed):
    kw = [dict(), dict(h0=True), dict(T=0.6), dict(L=4, M=3, V=7, B=9),
          dict(M=10, V=10, B=8), dict(dtype=synth.DT_BF16), dict(gru_bias=False, head_bias=False),
          dict(L=2, M=5, B=11)][seed]
    assert bruteforce_mismatch(small(100 + seed, **kw)) is None


@pytest.mark.parametrize("k", [1, 2, 3])
def test_bruteforce_top_b_with_branching_cap(k):
    assert bruteforce_mismatch(small(7 + k, L=4, M=4, V=9, B=7), max_children=k) is None


def test_bruteforce_slice_normalisation():
    assert bruteforce_mismatch(small(41, T=1.3), norm_slice=True) is None


def _zero_head(wl):
    wl.weights.w_c = np.zeros_like(wl.weights.w_c)
    if wl.weights.b_c is not None:
        wl.weights.b_c = np.zeros_like(wl.weights.b_c)
    return wl


def factorized_mismatch(wl, norm_slice=False, max_children=0):
    out = run_oracle(wl, max_children=max_children,
                     norm_mode=oracle.NORM_SLICE if norm_slice else oracle.NORM_TAIL)
    k = min(wl.M, wl.B) if max_children <= 0 else min(max_children, wl.M)
    toks, pars, deps, gs = indep.factorized_tree(wl.logits[0], wl.logits_dtype, wl.M, wl.B,
                                                 wl.T, k, norm_slice)
    n = out["n_nodes"]
    if n != len(toks):
        return f"n_nodes {n} vs {len(toks)}"
    if out["tokens"][:n].tolist() != toks or out["parents"][:n].tolist() != pars:
        return "topology differs"
    if out["depth"][:n].tolist() != deps:
        return "depth differs"
    if np.max(np.abs(out["scores"][:n] - np.array(gs))) > 1e-9:
        return "scores differ"
    return None


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("norm_slice", [False, True])
def test_zeroed_correction_is_factorized_tree(seed, norm_slice):
    wl = _zero_head(synth.random_small(200 + seed, batch=1, L=5, V=300, M=16, B=24,
                                       T=[0.0, 0.8, 1.5, 0.0][seed], d_e=8, d_h=6, h0=True))
    assert factorized_mismatch(wl, norm_slice) is None


def test_zeroed_correction_tiny_workload():
    wl = _zero_head(synth.tiny())
    assert factorized_mismatch(wl) is None


def test_path_independent_correction_closed_form():
    # W_ih = W_hh = 0, no GRU bias, h0 = 0: the state stays 0, so delta(v) = E[v].b_c
    # at every node; with M = V the tree is the factorised tree of X + E b_c.
    wl = synth.random_small(300, batch=1, L=4, V=12, M=12, B=10, T=0.0, d_e=5, d_h=4,
                            gru_bias=False, emb_std=1.0, w_scale=1.0)
    w = wl.weights
    w.w_ih = np.zeros_like(w.w_ih)
    w.w_hh = np.zeros_like(w.w_hh)
    out = run_oracle(wl)
    shift = w.emb.astype(np.float64) @ w.b_c.astype(np.float64)
    Xs = (wl.logits[0].astype(np.float64) + shift[None, :]).astype(np.float32)
    toks, pars, deps, gs = indep.factorized_tree(Xs, synth.DT_F32, wl.M, wl.B, wl.T, wl.B)
    n = out["n_nodes"]
    assert out["tokens"][:n].tolist() == toks
    assert out["parents"][:n].tolist() == pars
    np.testing.assert_allclose(out["scores"][:n], gs, atol=1e-6)


@pytest.mark.parametrize("seed", range(4))
def test_k1_budget_L_is_greedy_chain(seed):
    wl = synth.random_small(400 + seed, batch=1, L=6, V=50, M=8, B=6, T=0.0, d_e=7, d_h=5,
                            h0=bool(seed % 2), emb_std=1.0, w_scale=0.8)
    out = run_oracle(wl, max_children=1)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights,
                           None if wl.h0 is None else wl.h0[0], wl.M, wl.T)
    chain = indep.greedy_chain(sc, wl.L)
    assert out["n_nodes"] == wl.L
    assert out["tokens"][: wl.L].tolist() == chain
    assert out["parents"][: wl.L].tolist() == list(range(-1, wl.L - 1))


def test_budget_one_is_first_greedy_step():
    wl = synth.random_small(450, batch=1, L=5, V=40, M=6, B=1, T=0.0, d_e=5, d_h=4)
    out = run_oracle(wl)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, None, wl.M, wl.T)
    assert out["n_nodes"] == 1
    assert out["tokens"][0] == indep.greedy_chain(sc, 1)[0]
    assert out["parents"][0] == -1


def test_tiny_workload_chain_with_k1():
    wl = synth.tiny()
    wl.B = wl.L
    out = run_oracle(wl, max_children=1)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, None, wl.M, wl.T)
    assert out["tokens"][: wl.L].tolist() == indep.greedy_chain(sc, wl.L)


@pytest.mark.parametrize("seed", range(4))
def test_frontier_builder_recovers_heap_tree(seed):
    wl = small(500 + seed, L=4, V=12, M=5, B=8, h0=True)
    out = run_oracle(wl)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, wl.h0[0], wl.M, wl.T)
    got = indep.frontier_tree(sc, wl.B, min(wl.M, wl.B))
    assert got == set(oracle_paths(out))


@pytest.mark.parametrize("seed", range(5))
def test_invariants(seed):
    wl = synth.random_small(600 + seed, batch=1, L=6, V=80, M=10, B=20, T=0.9, d_e=9, d_h=7,
                            h0=True)
    for norm in (oracle.NORM_TAIL, oracle.NORM_SLICE):
        out = run_oracle(wl, norm_mode=norm, pos_offset=17)
        n = out["n_nodes"]
        assert n == wl.B
        errs = check_tree_valid(out["tokens"], out["parents"], out["depth"],
                                out["position_ids"], out["mask"], out["scores"], n, wl.B, 17)
        assert errs == []
        assert np.all(out["scores"][:n] <= 0)
    # normalisation identities of the slot log-probs
    w = wl.weights
    from helpers import weight_dict
    for norm in (oracle.NORM_TAIL, oracle.NORM_SLICE):
        m = ref._Model(oracle.widen(wl.logits[0], wl.logits_dtype), w.emb, w.dtype,
                       weight_dict(w), wl.M, 0.9, norm)
        S = np.random.default_rng(seed).standard_normal(w.d_h)
        for d in range(1, wl.L + 1):
            ell, live = m.slot_logprobs(S, d)
            assert np.all(ell[live] <= 0)
            mass = np.sum(np.exp(ell[live]))
            if norm == oracle.NORM_SLICE:
                assert mass == pytest.approx(1.0, abs=1e-12)
            else:
                assert mass < 1.0
                # tail share = exp(R - logZ); logZ = z_m - ell_m for any live m
                mm = int(np.flatnonzero(live)[0])
                xz = (m.xc[d - 1][mm] + m.Ec[d - 1][mm] @ (m.w_c @ S + m.b_c)) / 0.9
                logZ = xz - ell[mm]
                assert mass + math.exp(m.R[d - 1] - logZ) == pytest.approx(1.0, abs=1e-12)


def test_small_candidate_tree_pads():
    # k = 1 and L = 3 gives a 3-node candidate tree; budget 5 leaves 2 padding rows
    wl = small(700, L=3, B=5)
    out = run_oracle(wl, max_children=1, pos_offset=4)
    assert out["n_nodes"] == 3
    assert check_tree_valid(out["tokens"], out["parents"], out["depth"], out["position_ids"],
                            out["mask"], out["scores"], 3, 5, 4) == []


def test_temperature_zero_equals_one():
    a = small(800, T=0.0, h0=True)
    b = small(800, T=1.0, h0=True)
    oa, ob = run_oracle(a), run_oracle(b)
    for key in ("tokens", "parents", "depth", "mask"):
        np.testing.assert_array_equal(oa[key], ob[key])
    np.testing.assert_array_equal(oa["scores"], ob["scores"])


def test_full_vocab_tail_equals_slice():
    wl = small(900, M=10, V=10, B=9, T=0.7)
    ot = run_oracle(wl, norm_mode=oracle.NORM_TAIL)
    os_ = run_oracle(wl, norm_mode=oracle.NORM_SLICE)
    np.testing.assert_array_equal(ot["tokens"], os_["tokens"])
    np.testing.assert_allclose(ot["scores"][:9], os_["scores"][:9], atol=1e-12)


def test_nonfinite_logits_flag_tree():
    wl = small(1000)
    x = wl.logits.copy()
    x[0, 1, 3] = np.nan
    wl.logits = x
    out = run_oracle(wl)
    assert out["status"] == oracle.TREE_NONFINITE and out["n_nodes"] == 0
    x[0, 1, 3] = np.inf
    assert run_oracle(wl)["status"] == oracle.TREE_NONFINITE


def test_dead_slots_never_become_nodes():
    wl = small(1100, V=10, M=6, B=12)
    x = wl.logits.copy()
    x[0, 0, :] = -np.inf
    x[0, 0, [2, 5]] = [1.0, 0.5]      # only two live tokens at depth 1
    wl.logits = x
    out = run_oracle(wl)
    n = out["n_nodes"]
    d1 = out["tokens"][:n][out["depth"][:n] == 1]
    assert sorted(d1.tolist()) == [2, 5]


def _golden_case(c):
    V, de, dh = c["V"], c["d_e"], c["d_h"]
    X = np.log(np.array(c["logits_probs"], np.float64)).astype(np.float32)
    w = dict(w_ih=np.array(c["w_ih"], np.float32), w_hh=np.array(c["w_hh"], np.float32),
             b_ih=None, b_hh=None, w_c=np.array(c["w_c"], np.float32),
             b_c=np.array(c["b_c"], np.float32), dtype=oracle.DT_F32)
    emb = np.array(c["emb"], np.float32)
    return oracle.build_tree(X, emb, oracle.DT_F32, w, np.array(c["h0"], np.float64), c["M"],
                             c["B"], c["T"])


def golden_mismatch():
    cases = json.load(open(GOLDEN))["cases"]
    for c in cases:
        out = _golden_case(c)
        e = c["expect"]
        n = len(e["tokens"])
        if out["n_nodes"] != n:
            return c["name"] + ": n_nodes"
        for key in ("tokens", "parents", "depth"):
            if out[key][:n].tolist() != e[key]:
                return c["name"] + ": " + key
        if out["mask"][:n, :n].tolist() != e["mask"]:
            return c["name"] + ": mask"
        if np.max(np.abs(out["scores"][:n] - np.log(e["scores_probs"]))) > 1e-6:
            return c["name"] + ": scores"
    return None


def test_golden_hand_trees():
    assert golden_mismatch() is None


# ---------------------------------------------------------------------------
# planted mistakes: each must make at least one pin fail
# ---------------------------------------------------------------------------

def _pins_fail():
    bad = []
    try:
        bad.append(golden_mismatch())
        for s in range(3):
            bad.append(bruteforce_mismatch(small(100 + s, h0=True, T=[0.0, 0.6, 1.0][s])))
        bad.append(factorized_mismatch(_zero_head(synth.random_small(
            210, batch=1, L=4, V=200, M=12, B=16, T=0.0, d_e=8, d_h=6))))
    except Exception as e:          # a crash also counts as a failed pin
        bad.append(repr(e))
    return any(b is not None for b in bad)


MUTANTS = {
    "gru_r_z_swapped": "swap",
    "head_bias_dropped": "nobias",
    "correction_sign": "sign",
    "head_transposed": "transpose",
    "tail_dropped": "notail",
    "temperature_ignored": "notau",
    "min_heap": "minheap",
    "state_not_advanced": "nostate",
}


@pytest.mark.parametrize("mutant", list(MUTANTS))
def test_planted_mistake_is_caught(mutant, monkeypatch):
    kind = MUTANTS[mutant]
    orig_slot = ref._Model.slot_logprobs
    orig_gru = ref.gru_cell

    if kind == "swap":
        def bad_gru(h, xs, w_ih, w_hh, b_ih, b_hh):
            d = h.shape[0]
            perm = np.r_[d:2 * d, 0:d, 2 * d:3 * d]
            return orig_gru(h, xs, w_ih[perm], w_hh[perm],
                            None if b_ih is None else b_ih[perm],
                            None if b_hh is None else b_hh[perm])
        monkeypatch.setattr(ref, "gru_cell", bad_gru)
    elif kind == "nostate":
        monkeypatch.setattr(ref, "gru_cell", lambda h, xs, *a: np.repeat(h[None], len(xs), 0))
    elif kind in ("nobias", "sign", "transpose", "notail", "notau"):
        def bad_slot(self, S, d):
            if kind == "nobias":
                saved, self.b_c = self.b_c, None
                try:
                    return orig_slot(self, S, d)
                finally:
                    self.b_c = saved
            if kind == "transpose":
                saved = self.w_c
                self.w_c = np.ascontiguousarray(saved.T) if saved.shape[0] == saved.shape[1] \
                    else saved[:, ::-1]
                try:
                    return orig_slot(self, S, d)
                finally:
                    self.w_c = saved
            if kind == "notail":
                saved, self.norm_mode = self.norm_mode, ref.NORM_SLICE
                try:
                    return orig_slot(self, S, d)
                finally:
                    self.norm_mode = saved
            if kind == "notau":
                saved, self.tau = self.tau, 1.0
                try:
                    return orig_slot(self, S, d)
                finally:
                    self.tau = saved
            # sign
            saved = self.Ec[d - 1]
            self.Ec[d - 1] = -saved
            try:
                return orig_slot(self, S, d)
            finally:
                self.Ec[d - 1] = saved
        monkeypatch.setattr(ref._Model, "slot_logprobs", bad_slot)
    elif kind == "minheap":
        import heapq as hq

        class FlippedHeap:
            @staticmethod
            def heappush(h, e):
                hq.heappush(h, (-e[0],) + e[1:])

            @staticmethod
            def heappop(h):
                e = hq.heappop(h)
                return (-e[0],) + e[1:]
        monkeypatch.setattr(ref, "heapq", FlippedHeap)
    assert _pins_fail(), f"planted mistake {mutant} went unnoticed"

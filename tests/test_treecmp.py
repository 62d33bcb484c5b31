"""The tie-aware tree comparison itself, on oracle trees and planted deviations (CPU only).

The comparison must accept the oracle's own tree, a permutation of a near-tie
band and a near-tied substitute at a top-k cut, and must reject a node moved
across a decisive gap, a clearly worse substitute and a wrong parent.
"""
import json
import os

import numpy as np
import pytest

import indep
import oracle
import treecmp
from helpers import rescore, run_oracle
from paper_2607_08642_amd import synth

TIES = os.path.join(os.path.dirname(__file__), "golden", "tie_trees.json")


def as_got(paths, B, rs, pos_offset=0, tie_tol=0.0):
    """An emitted tree (host arrays) holding `paths` in the given pop order,
    scored by re-scoring."""
    n = len(paths)
    index = {p: i for i, p in enumerate(paths)}
    tok = np.full(B, -1, np.int32)
    par = np.full(B, -1, np.int32)
    dep = np.zeros(B, np.int32)
    mask = np.zeros((B, B), np.uint8)
    for i, p in enumerate(paths):
        tok[i] = p[-1]
        par[i] = index[p[:-1]] if len(p) > 1 else -1
        dep[i] = len(p)
        mask[i, i] = 1
        if par[i] >= 0:
            mask[i] |= mask[par[i]]
    g, valid = rs(tok, par, n, tie_tol)
    assert valid
    sc = np.full(B, -np.inf, np.float32)
    sc[:n] = g
    return dict(tokens=tok, parents=par, depth=dep, position_ids=pos_offset + dep, mask=mask,
                scores=sc, n_nodes=n, status=0)


def tie_case():
    c = json.load(open(TIES))["cases"][0]
    X = np.log(np.array(c["logits_probs"], np.float64)).astype(np.float32)
    w = synth.Weights(np.zeros((4, 1), np.float32), np.zeros((3, 1), np.float32),
                      np.zeros((3, 1), np.float32), None, None, np.zeros((1, 1), np.float32),
                      np.zeros(1, np.float32), synth.DT_F32, 4, 1, 1)
    return synth.Workload("ties", X[None], synth.DT_F32, None, w, 2, 4, c["B"], 0.0, 1)


def rs_for(wl, **kw):
    return lambda tok, par, n, tie_tol: rescore(wl, 0, tok, par, n, tie_tol=tie_tol, **kw)


def paths_of(ref):
    return treecmp.tree_paths(ref["tokens"], ref["parents"], ref["n_nodes"])


def test_oracle_tree_is_exact():
    wl = tie_case()
    ref = run_oracle(wl)
    got = as_got(paths_of(ref), wl.B, rs_for(wl))
    kind, err, _ = treecmp.compare(ref, got, rs_for(wl), 1e-4)
    assert kind == "exact" and err < 1e-6


def test_tied_band_may_permute():
    wl = tie_case()
    ref = run_oracle(wl)
    p = paths_of(ref)
    p[4], p[5] = p[5], p[4]               # two tied depth-2 children of pop 0
    p[6], p[8] = p[8], p[6]               # tied children of different parents
    kind, _, n_exact = treecmp.compare(ref, as_got(p, wl.B, rs_for(wl)), rs_for(wl), 1e-4)
    assert kind == "banded" and n_exact == 0


def test_clearly_worse_substitute_is_rejected():
    wl = tie_case()
    ref = run_oracle(wl)
    p = paths_of(ref)
    p[9] = (2, 0)                          # .05 in place of a .075 node
    with pytest.raises(AssertionError):
        treecmp.compare(ref, as_got(p, wl.B, rs_for(wl)), rs_for(wl), 1e-4)


def random_case():
    wl = synth.random_small(71, batch=1, L=4, V=30, M=6, B=12, T=0.9, d_e=6, d_h=5, h0=True,
                            logit_scale=1.0, emb_std=0.8, w_scale=0.8)
    return wl, run_oracle(wl, max_children=3)


def test_decisive_tree_swap_is_rejected():
    wl, ref = random_case()
    assert ref["min_gap"] > 1e-4
    p = paths_of(ref)
    # swap two pops that are not ancestor and descendant
    i, j = next((i, j) for i in range(1, len(p)) for j in range(i + 1, len(p))
                if p[j][:len(p[i])] != p[i])
    p[i], p[j] = p[j], p[i]
    with pytest.raises(AssertionError):
        treecmp.compare(ref, as_got(p, wl.B, rs_for(wl, max_children=3)),
                        rs_for(wl, max_children=3), 1e-4)


def test_wide_band_permutation_and_cross_band_move():
    # an artificially wide gap threshold makes near-tie bands of a tie-free tree
    wl, ref = random_case()
    n = ref["n_nodes"]
    s = ref["scores"][:n]
    pops = np.sort(s[:-1] - s[1:])
    gap = float(pops[2]) * 1.0001             # the three smallest pop gaps join bands
    band, crossing = treecmp.bands(s, n, wl.B, ref["excluded"], gap)
    soft = treecmp.soft_nodes(ref, n, gap)
    p = paths_of(ref)
    rs = rs_for(wl, max_children=3)
    # a band of two unrelated, non-soft pops that does not reach the boundary
    cand = [(i, i + 1) for i in range(n - 1) if band[i] == band[i + 1]
            and not soft[i] and not soft[i + 1] and p[i + 1][:len(p[i])] != p[i]
            and not (crossing and band[i] == band[-1]) and np.sum(band == band[i]) == 2]
    assert cand, "no permutable band in this case"
    i, j = cand[0]
    q = list(p)
    q[i], q[j] = q[j], q[i]
    kind, _, _ = treecmp.compare(ref, as_got(q, wl.B, rs), rs, 1e-4, gap=gap)
    assert kind == "banded"
    # moving a node into another band is rejected
    k = next(k for k in range(n) if band[k] != band[i] and p[k][:len(p[i])] != p[i]
             and p[i][:len(p[k])] != p[k] and abs(s[k] - s[i]) > gap)
    q = list(p)
    q[i], q[k] = q[k], q[i]
    with pytest.raises(AssertionError):
        treecmp.compare(ref, as_got(q, wl.B, rs), rs, 1e-4, gap=gap)


def test_near_tied_substitute_at_topk_cut():
    # a child whose log-prob lies within the threshold of its expansion's cut
    # may be replaced by the best sibling that was cut off
    wl, ref = random_case()
    n = ref["n_nodes"]
    margin = ref["ell"][:n] - ref["ell_out"][:n]
    leaves = [i for i in range(n) if i not in set(ref["parents"][:n].tolist())]
    i = min(leaves, key=lambda x: margin[x])
    gap = float(margin[i]) * 1.5
    p = paths_of(ref)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, wl.h0[0], wl.M, wl.T)
    S = sc.h0
    for tok in p[i][:-1]:
        S = sc.step(S, tok)
    ranked = sc.ranked_children(S, len(p[i]), wl.M)
    cut_tok = ranked[3][0]                       # k = 3: the best child cut off
    q = list(p)
    q[i] = p[i][:-1] + (cut_tok,)
    rs = rs_for(wl, max_children=3)
    got = as_got(q, wl.B, rs, tie_tol=gap)
    kind, _, _ = treecmp.compare(ref, got, rs, 1e-4, gap=gap)
    assert kind == "banded"
    with pytest.raises(AssertionError):          # at the default threshold it is a mismatch
        treecmp.compare(ref, got, rs, 1e-4)


def test_wrong_parent_is_rejected():
    wl = tie_case()
    ref = run_oracle(wl)
    got = as_got(paths_of(ref), wl.B, rs_for(wl))
    got["parents"] = got["parents"].copy()
    got["parents"][4] = 1                  # (0,0) re-hung under token 1: node (1,0) instead
    got["mask"][4] = 0
    got["mask"][4, [1, 4]] = 1
    with pytest.raises(AssertionError):
        treecmp.compare(ref, got, rs_for(wl), 1e-4)


def test_moved_subtree_is_rejected():
    wl, ref = random_case()
    got = as_got(paths_of(ref), wl.B, rs_for(wl, max_children=3))
    n = ref["n_nodes"]
    i = next(i for i in range(n) if ref["parents"][i] >= 1)
    got["parents"] = got["parents"].copy()
    got["parents"][i] = ref["parents"][i] - 1   # hung under the previous pop
    with pytest.raises(AssertionError):
        treecmp.compare(ref, got, rs_for(wl, max_children=3), 1e-4)

"""Pins of the oracle's Domino-head scorer (section 2.3: delta = W_2 SiLU(W_1 [H_d; S]),
rank-r bottleneck, W_2's rows gathered for the depth's slice).

* a hand-derived tree: one-unit state, rank 1, a GRU that halves the state;
* W_2 = 0: no correction, so the tree is the Marg tree;
* W_1's state half = 0: the correction depends on the depth only, so the tree
  is DDTree's heap over per-depth menus from an independent torch scorer
  (full-vocabulary log-softmax, torch.nn.functional.silu);
* brute force: the oracle's tree is the top-B set of every path of the
  k-restricted candidate tree scored by that torch scorer with torch's GRUCell.
"""
import math

import numpy as np
import pytest

import indep
from helpers import oracle, weight_dict
from paper_2607_08642_amd import synth


def _same_tree(out, toks, pars, deps, gs, atol=1e-9):
    n = out["n_nodes"]
    assert n == len(toks)
    assert out["tokens"][:n].tolist() == toks
    assert out["parents"][:n].tolist() == pars
    assert out["depth"][:n].tolist() == deps
    np.testing.assert_allclose(out["scores"][:n], gs, atol=atol)


def _run(wl, head, H, t=0, **kw):
    w = weight_dict(wl.weights)
    w.update(w1=head.w1, w2=head.w2)
    return oracle.build_tree(wl.logits[t], wl.weights.emb, wl.weights.dtype, w,
                             None if wl.h0 is None else wl.h0[t], wl.M, wl.B, wl.T,
                             logits_dtype=wl.logits_dtype, scorer=oracle.SCORER_HEAD,
                             H=H[t], **kw)


def _case(seed, **kw):
    args = dict(batch=1, L=4, V=40, M=8, B=12, T=0.8, d_e=6, d_h=5, emb_std=0.8, w_scale=0.8)
    args.update(kw)
    wl = synth.random_small(seed, **args)
    d_H, rank = 7, 6
    head = synth.domino_head(seed, args["V"], d_H, args["d_h"], rank, wl.weights.dtype,
                             w1_scale=0.9, w2_scale=1.2)
    H = synth.hidden_states(seed, 1, args["L"], d_H, wl.weights.dtype)
    return wl, head, H


def test_hand_derived_tree():
    # d_h = d_H = rank = 1, V = M = 3, tau = 1, zero logits, h0 = 0.5.
    # W_ih = W_hh = 0 and no GRU bias: r = z = 1/2, n = 0, so a step halves the state.
    # W_1 = [1, 2], W_2 = [1, -2, 0.5]^T, H = [0, 1].
    # depth 1: u = 0 + 2 * 0.5 = 1;   y = SiLU(1)   = 0.7310585786300049
    # depth 2: u = 1 + 2 * 0.25 = 1.5; y = SiLU(1.5) = 1.2263617142904655
    # ell = delta - LSE(delta) with delta = (y, -2y, y/2) (no token outside the slice)
    z32 = lambda *s: np.zeros(s, np.float32)
    w = dict(w_ih=z32(3, 1), w_hh=z32(3, 1), b_ih=None, b_hh=None, w_c=z32(1, 1), b_c=None,
             dtype=oracle.DT_F32, w1=np.array([[1.0, 2.0]], np.float32),
             w2=np.array([[1.0], [-2.0], [0.5]], np.float32))
    out = oracle.build_tree(z32(2, 3), z32(3, 1), oracle.DT_F32, w, np.array([0.5], np.float32),
                            3, 3, 1.0, scorer=oracle.SCORER_HEAD,
                            H=np.array([[0.0], [1.0]], np.float32))
    l1 = [-0.590777306013437, -2.7839530419034517, -0.9563065953284395]
    l2 = [-0.4490808631639902, -4.128166006035387, -1.0622617203092228]
    _same_tree(out, [0, 2, 0], [-1, -1, 0], [1, 1, 2], [l1[0], l1[2], l1[0] + l2[0]], atol=1e-13)


@pytest.mark.parametrize("seed", range(3))
def test_zero_w2_is_the_marg_tree(seed):
    wl, head, H = _case(1100 + seed, h0=bool(seed % 2))
    head.w2 = np.zeros_like(head.w2)
    a = _run(wl, head, H)
    w = wl.weights
    b = oracle.build_tree(wl.logits[0], w.emb, w.dtype, weight_dict(w),
                          None if wl.h0 is None else wl.h0[0], wl.M, wl.B, wl.T,
                          logits_dtype=wl.logits_dtype, scorer=oracle.SCORER_MARG)
    for key in ("tokens", "parents", "depth"):
        np.testing.assert_array_equal(a[key], b[key])
    np.testing.assert_allclose(a["scores"][: a["n_nodes"]], b["scores"][: b["n_nodes"]], atol=1e-12)


@pytest.mark.parametrize("seed", range(3))
def test_state_free_head_is_a_menu_heap(seed):
    wl, head, H = _case(1200 + seed, h0=True, T=[0.0, 0.7, 1.4][seed])
    w1 = head.w1.copy()
    w1[:, head.d_H:] = 0
    head.w1 = w1
    out = _run(wl, head, H)
    sc = indep.HeadTorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, head, H[0],
                               wl.h0[0], wl.M, wl.T)
    k = min(wl.M, wl.B)
    _same_tree(out, *indep.menu_tree(sc, wl.B, k, sc.h0), atol=1e-9)


@pytest.mark.parametrize("seed", range(6))
def test_bruteforce_top_b(seed):
    kw = [dict(), dict(h0=True), dict(T=0.0), dict(dtype=synth.DT_BF16),
          dict(L=3, M=5, V=12, B=9, gru_bias=False), dict(L=2, M=6, B=10, h0=True)][seed]
    args = dict(L=3, V=10, M=4, B=7)
    args.update(kw)
    wl, head, H = _case(1300 + seed, **args)
    k = min(wl.M, wl.B)
    out = _run(wl, head, H)
    sc = indep.HeadTorchScorer(wl.logits[0], wl.logits_dtype, wl.weights, head, H[0],
                               None if wl.h0 is None else wl.h0[0], wl.M, wl.T)
    allp = indep.enumerate_paths(sc, k)
    top, gap = indep.top_b_paths(allp, wl.B)
    assert gap > 1e-9, "seed has ties at the budget boundary"
    got = indep.tree_paths(out["tokens"], out["parents"], out["n_nodes"])
    assert set(got) == top
    for p, g in zip(got, out["scores"][: out["n_nodes"]]):
        assert abs(allp[p] - g) < 1e-10


def test_head_differs_from_the_linear_head():
    wl, head, H = _case(1400, h0=True)
    a = _run(wl, head, H)
    w = wl.weights
    b = oracle.build_tree(wl.logits[0], w.emb, w.dtype, weight_dict(w), wl.h0[0], wl.M, wl.B,
                          wl.T, logits_dtype=wl.logits_dtype)
    assert not np.allclose(a["scores"][: a["n_nodes"]], b["scores"][: b["n_nodes"]])
    assert math.isfinite(a["scores"][0])

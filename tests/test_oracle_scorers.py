"""Pins of the oracle's ablation-arm scorers (Appendix D, the three arms).

* Marg: a depth's slice scored from the marginal logits alone, whatever the
  correction head holds -> DDTree's factorised tree over full-vocabulary
  log-softmax menus (an independent torch implementation).
* Cond-static: the correction once per depth along Domino's greedy chain ->
  an independent builder from the definition (torch GRUCell and full-vocabulary
  log-softmax, menus shared per depth), the greedy chain itself at k = 1, and
  the DominoTree tree whenever the correction does not depend on the path.
"""
import numpy as np
import pytest

import indep
from helpers import oracle, run_oracle
from paper_2607_08642_amd import synth


def _same_tree(out, toks, pars, deps, gs, atol=1e-9):
    n = out["n_nodes"]
    assert n == len(toks)
    assert out["tokens"][:n].tolist() == toks
    assert out["parents"][:n].tolist() == pars
    assert out["depth"][:n].tolist() == deps
    np.testing.assert_allclose(out["scores"][:n], gs, atol=atol)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("norm_slice", [False, True])
def test_marg_is_factorised_tree_whatever_the_head(seed, norm_slice):
    wl = synth.random_small(600 + seed, batch=1, L=5, V=300, M=16, B=24,
                            T=[0.0, 0.8, 1.5, 0.6][seed], d_e=8, d_h=6, h0=True,
                            emb_std=1.0, w_scale=1.0)
    out = run_oracle(wl, scorer=oracle.SCORER_MARG,
                     norm_mode=oracle.NORM_SLICE if norm_slice else oracle.NORM_TAIL)
    k = min(wl.M, wl.B)
    _same_tree(out, *indep.factorized_tree(wl.logits[0], wl.logits_dtype, wl.M, wl.B, wl.T, k,
                                           norm_slice))


@pytest.mark.parametrize("seed", range(4))
def test_static_matches_independent_builder(seed):
    wl = synth.random_small(700 + seed, batch=1, L=5, V=200, M=12, B=20,
                            T=[0.0, 0.7, 1.3, 1.0][seed], d_e=7, d_h=5, h0=bool(seed % 2),
                            emb_std=1.0, w_scale=0.8)
    k = [0, 3, 0, 5][seed]
    out = run_oracle(wl, scorer=oracle.SCORER_STATIC, max_children=k)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights,
                           None if wl.h0 is None else wl.h0[0], wl.M, wl.T)
    kk = min(wl.M, wl.B) if k <= 0 else min(k, wl.M)
    _same_tree(out, *indep.static_tree(sc, wl.B, kk), atol=1e-9)


@pytest.mark.parametrize("seed", range(3))
def test_static_chain_is_the_greedy_chain(seed):
    wl = synth.random_small(800 + seed, batch=1, L=6, V=50, M=8, B=6, T=0.0, d_e=7, d_h=5,
                            h0=bool(seed % 2), emb_std=1.0, w_scale=0.8)
    out = run_oracle(wl, scorer=oracle.SCORER_STATIC, max_children=1)
    sc = indep.TorchScorer(wl.logits[0], wl.logits_dtype, wl.weights,
                           None if wl.h0 is None else wl.h0[0], wl.M, wl.T)
    assert out["tokens"][: wl.L].tolist() == indep.greedy_chain(sc, wl.L)
    # ... which DominoTree's k = 1 tree walks too, with the same scores
    cond = run_oracle(wl, max_children=1)
    np.testing.assert_array_equal(out["tokens"], cond["tokens"])
    np.testing.assert_allclose(out["scores"][: wl.L], cond["scores"][: wl.L], atol=1e-12)


def test_static_equals_cond_when_the_correction_is_path_independent():
    # W_ih = W_hh = 0, no GRU bias, h0 = 0: every path state is 0, so the greedy
    # chain's correction is every node's correction
    wl = synth.random_small(900, batch=1, L=4, V=40, M=10, B=16, T=0.7, d_e=5, d_h=4,
                            gru_bias=False, emb_std=1.0, w_scale=1.0)
    w = wl.weights
    w.w_ih = np.zeros_like(w.w_ih)
    w.w_hh = np.zeros_like(w.w_hh)
    a = run_oracle(wl, scorer=oracle.SCORER_STATIC)
    b = run_oracle(wl)
    for key in ("tokens", "parents", "depth"):
        np.testing.assert_array_equal(a[key], b[key])
    np.testing.assert_allclose(a["scores"][: a["n_nodes"]], b["scores"][: b["n_nodes"]], atol=1e-12)


def test_scorers_differ_on_a_path_dependent_model():
    # the three arms are different functions: on a model whose correction
    # depends on the path, at least one pair of trees differs
    wl = synth.random_small(950, batch=1, L=5, V=300, M=16, B=24, T=0.8, d_e=8, d_h=6,
                            h0=True, emb_std=1.0, w_scale=1.5)
    trees = [run_oracle(wl, scorer=s) for s in (oracle.SCORER_COND, oracle.SCORER_MARG,
                                                  oracle.SCORER_STATIC)]
    sig = [tuple(t["tokens"].tolist()) + tuple(np.round(t["scores"], 9).tolist()) for t in trees]
    assert len(set(sig)) == 3

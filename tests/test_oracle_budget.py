"""Pins of the oracle's adaptive budget (CaDDTree's stopping rule, section 2.5,
carried into the conditional pop loop, section 3.4; CPU only).

theta(n) = (1 + Phi(n)) / (C_d + C_v(n)), Phi(n) = sum of exp(g_s) over the
first n pops; the loop stops the first time theta does not improve.

* hand-derived stop points on the factorised golden tree (pop probabilities
  .5, .3, .25, .15, .1, .05) under a quadratic and a linear verify cost;
* CaDDTree's unimodality: with a convex C_v the greedy stop equals the global
  argmax of theta over the fixed-budget tree's pop sequence, computed apart;
* limits: a flat C_v runs to the cap, a steep one stops at 0 nodes, and a
  non-convex bump stops at the first non-improvement, not the argmax.
"""
import math

import numpy as np
import pytest

import oracle
from helpers import run_oracle
from paper_2607_08642_amd import synth


def golden_factorized(B):
    # rows log(.5 .25 .125 .125) and log(.1 .6 .2 .1), M = 2, zero correction:
    # full pop sequence (0) .5, (0,1) .3, (1) .25, (1,1) .15, (0,2) .1, (1,2) .05
    X = np.log(np.array([[0.5, 0.25, 0.125, 0.125], [0.1, 0.6, 0.2, 0.1]])).astype(np.float32)
    z = np.zeros
    w = dict(w_ih=z((3, 1), np.float32), w_hh=z((3, 1), np.float32), b_ih=None, b_hh=None,
             w_c=z((1, 1), np.float32), b_c=z(1, np.float32), dtype=oracle.DT_F32)
    emb = z((4, 1), np.float32)
    return lambda costs: oracle.build_tree(X, emb, oracle.DT_F32, w, None, 2, B, 0.0,
                                           budget_costs=costs)


def test_hand_derived_stop_quadratic_cost():
    # C_d = 1, C_v(n) = 0.02 n^2: theta = 1, 1.5/1.02, 1.8/1.08, 2.05/1.18, 2.2/1.32
    # = 1, 1.4706, 1.6667, 1.7373, 1.6667: the fourth pop does not improve -> 3 nodes
    build = golden_factorized(6)
    out = build((1.0, [0.02 * n * n for n in range(7)]))
    assert out["n_nodes"] == 3
    assert out["tokens"][:3].tolist() == [0, 1, 1]
    assert out["parents"][:3].tolist() == [-1, 0, -1]
    np.testing.assert_allclose(np.exp(out["scores"][:3]), [0.5, 0.3, 0.25], atol=1e-6)
    assert out["tokens"][3] == -1 and out["depth"][3] == 0      # padding past the stop
    # the stop decision's margin: (theta(3) - theta(4)) / theta(3)
    budget = [v for k, v in out["gaps"] if k == "budget"]
    assert len(budget) == 4
    assert min(budget) == pytest.approx((2.05 / 1.18 - 2.2 / 1.32) / (2.05 / 1.18), rel=1e-5)


def test_hand_derived_stop_linear_cost():
    # C_v(n) = 0.05 n: theta = 1, 1.4286, 1.6364, 1.7826, 1.8333, 1.84, 2.35/1.3 = 1.8077
    # -> 5 nodes; the sixth pop (.05) does not improve
    out = golden_factorized(6)((1.0, [0.05 * n for n in range(7)]))
    assert out["n_nodes"] == 5
    assert out["tokens"][:5].tolist() == [0, 1, 1, 1, 2]
    assert out["parents"][:5].tolist() == [-1, 0, -1, 2, 0]


def test_flat_cost_runs_to_cap_and_steep_cost_stops_empty():
    build = golden_factorized(6)
    full = build(None)
    flat = build((1.0, [0.5] * 7))
    assert flat["n_nodes"] == full["n_nodes"] == 6
    for k in ("tokens", "parents", "depth", "mask"):
        np.testing.assert_array_equal(flat[k], full[k])
    steep = build((1.0, [0.0] + [10.0] * 6))       # theta(1) = 1.5/11 < theta(0) = 1
    assert steep["n_nodes"] == 0 and (steep["tokens"] == -1).all()


def test_first_non_improvement_not_argmax():
    # a non-convex C_v: one expensive node then flat -- theta(1) = 1.5/1.6 < 1 stops at
    # 0 nodes, although theta(6) = 2.35/1.6 is the global maximum
    out = golden_factorized(6)((1.0, [0.0] + [0.6] * 6))
    assert out["n_nodes"] == 0


def theta_argmax(scores, c_d, c_v):
    """Global argmax of theta over n = 0..len(scores) (first maximum)."""
    phi = np.concatenate([[0.0], np.cumsum(np.exp(np.asarray(scores, np.float64)))])
    th = (1.0 + phi) / (c_d + np.asarray(c_v[:len(phi)], np.float64))
    return int(np.argmax(th)), th


@pytest.mark.parametrize("seed", range(6))
def test_greedy_stop_is_argmax_under_convex_cost(seed):
    rng = np.random.default_rng(seed)
    wl = synth.random_small(700 + seed, batch=1, L=5, V=60, M=8, B=24, T=[0.0, 0.7, 1.2][seed % 3],
                            d_e=8, d_h=6, h0=bool(seed % 2), logit_scale=1.0)
    full = run_oracle(wl, max_children=4)
    n_full = full["n_nodes"]
    c_d = float(rng.uniform(0.5, 2.0))
    a, c = float(rng.uniform(0.0, 0.01)), float(rng.uniform(0.0001, 0.0008))
    c_v = [a * n + c * n * n for n in range(wl.B + 1)]
    out = run_oracle(wl, max_children=4, budget_costs=(c_d, c_v))
    n_star, th = theta_argmax(full["scores"][:n_full], c_d, c_v)
    assert 0 < n_star < n_full      # the stop falls inside the tree (stops at 4..18 of 24)
    assert out["n_nodes"] == n_star, (out["n_nodes"], n_star, th)
    # the adaptive tree is the fixed-budget tree's first n* pops
    for k in ("tokens", "parents", "depth"):
        np.testing.assert_array_equal(out[k][:n_star], full[k][:n_star])
    assert (out["tokens"][n_star:] == -1).all()

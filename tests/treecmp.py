"""Tie-aware comparison of an emitted draft tree with the oracle's (host arrays only).

The heap pops nodes in score order with exact ties broken by insertion order
(Appendix B), so wherever consecutive oracle scores are more than GAP apart
the pop order is decided by the scores alone and both builders must agree node
for node.  Where scores lie within GAP of each other (a near-tie band) a GPU
tree computed in fp32 may order them differently, and where a band reaches
the budget boundary, or a child's log-prob lies within GAP of the top-k cut
of its parent's expansion, it may even hold a different, equally good node.
The comparison therefore checks:

* exact positions (a band of one, not at the boundary, not near a top-k cut,
  nor below such a node): the same node (its token path) at the same pop
  index, with the same parent index when the parent is an exact position too;
* bands of several nodes away from the boundary and the cuts: the same set of
  nodes at the band's pop indices (a permutation);
* every node, wherever it is: a valid top-k child of its parent under the
  tie tolerance, re-scored by the oracle along its own path, and the i-th
  re-scored score within GAP of the oracle's i-th score;
* the GPU's own scores within the score tolerance of the re-scored ones.
"""
from __future__ import annotations

import math
from typing import Callable, List

import numpy as np

GAP_TOL = 1e-4


def tree_paths(tokens, parents, n) -> List[tuple]:
    paths: List[tuple] = []
    for i in range(n):
        p = int(parents[i])
        paths.append((paths[p] if 0 <= p < i else ()) + (int(tokens[i]),))
    return paths


def bands(scores, n: int, B: int, excluded: float, gap: float):
    """Band index of every pop and whether the last band reaches the boundary."""
    band = np.zeros(n, np.int64)
    for i in range(1, n):
        band[i] = band[i - 1] + (1 if scores[i - 1] - scores[i] > gap else 0)
    # (an excluded entry exists when the budget, or the adaptive budget's stop,
    # ended the pops; an exhausted candidate tree leaves none)
    crossing = excluded > -math.inf and scores[n - 1] - excluded <= gap
    return band, crossing


def soft_nodes(ref, n: int, gap: float):
    """Nodes whose log-prob lies within gap of their expansion's top-k cut, and
    every node below one: another builder may keep a different child there.
    For the frontier builder also every node deeper than a depth whose top-W cut
    is that close: another lane may advance there."""
    soft = np.zeros(n, bool)
    cut_depths = [d for d, v in ref.get("frontier_cut", []) if v <= gap]
    shallow = min(cut_depths) if cut_depths else None
    for i in range(n):
        p = int(ref["parents"][i])
        soft[i] = (ref["ell"][i] - ref["ell_out"][i] <= gap) or (p >= 0 and soft[p]) or \
            (shallow is not None and int(ref["depth"][i]) > shallow)
    return soft


def compare(ref, got, rescore: Callable, tol: float, gap: float = GAP_TOL, B: int = None):
    """Compare one emitted tree `got` (dict of arrays: tokens, parents, depth,
    position_ids, mask, scores, n_nodes, status for this tree) with the oracle
    result `ref`.  rescore(tokens, parents, n, tie_tol) -> (g, valid).

    Returns (kind, max_score_error, n_exact_positions); kind is 'exact' (every
    field identical, scores within tol) or 'banded'.  Raises AssertionError.
    """
    B = len(ref["tokens"]) if B is None else B
    n = int(got["n_nodes"])
    assert n == ref["n_nodes"], f"n_nodes {n} vs {ref['n_nodes']}"
    if n == 0:
        return "exact", 0.0, 0
    sc = np.asarray(got["scores"], np.float64)[:n]
    fields = ("tokens", "parents", "depth", "position_ids")
    identical = all(np.array_equal(got[k], ref[k]) for k in fields) and \
        np.array_equal(got["mask"], ref["mask"])
    if ref["min_gap"] > gap:
        for k in fields:
            np.testing.assert_array_equal(got[k], ref[k], err_msg=k)
        np.testing.assert_array_equal(got["mask"], ref["mask"], err_msg="mask")
        err = float(np.max(np.abs(sc - ref["scores"][:n])))
        assert err <= tol, f"score error {err}"
        return "exact", err, n

    gp = tree_paths(got["tokens"], got["parents"], n)
    assert len(set(gp)) == n, "a node appears twice"
    # every node a valid (tie-tolerant) top-k child, re-scored along its own path
    g, valid = rescore(got["tokens"], got["parents"], n, gap)
    assert valid, "a node is not a top-k child of its parent's path"
    err = float(np.max(np.abs(sc - g)))
    assert err <= tol, f"score error {err} against the re-scored tree"
    s = np.asarray(ref["scores"][:n], np.float64)
    dev = np.abs(g - s)
    assert float(np.max(dev)) <= gap, \
        f"pop {int(np.argmax(dev))}: re-scored {g[np.argmax(dev)]} vs oracle {s[np.argmax(dev)]}"

    band, crossing = bands(s, n, B, ref["excluded"], gap)
    soft = soft_nodes(ref, n, gap)
    nb = int(band[-1]) + 1
    loose = np.zeros(nb, bool)
    for b in range(nb):
        members = band == b
        loose[b] = bool(np.any(soft[members])) or (crossing and b == nb - 1)
    exact_pos = np.array([not loose[band[i]] and np.sum(band == band[i]) == 1 for i in range(n)])
    rp = tree_paths(ref["tokens"], ref["parents"], n)
    for i in range(n):
        if exact_pos[i]:
            assert gp[i] == rp[i], f"pop {i}: node {gp[i]} vs oracle {rp[i]}"
            p = int(ref["parents"][i])
            if p < 0 or exact_pos[p]:
                assert int(got["parents"][i]) == p, f"pop {i}: parent {got['parents'][i]} vs {p}"
    for b in range(nb):
        idx = np.flatnonzero(band == b)
        if len(idx) > 1 and not loose[b]:
            assert {gp[i] for i in idx} == {rp[i] for i in idx}, \
                f"band {b} (pops {idx[0]}..{idx[-1]}): different nodes"
    if identical:
        return "exact", err, n
    return "banded", err, int(np.sum(exact_pos))

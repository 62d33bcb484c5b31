"""Shared test helpers: running the oracle on a synthetic workload, tree comparison."""
from __future__ import annotations

import math

import numpy as np

import oracle


def weight_dict(w):
    return dict(w_ih=w.w_ih, w_hh=w.w_hh, b_ih=w.b_ih, b_hh=w.b_hh, w_c=w.w_c, b_c=w.b_c,
                dtype=w.dtype)


def _oracle_inputs(wl, t, kw):
    """Weights dict and keyword arguments; a workload carrying Domino's own head
    (attributes head, H) adds w1, w2 and its tree's hidden states."""
    w = weight_dict(wl.weights)
    if kw.get("scorer") == oracle.SCORER_HEAD:
        w.update(w1=wl.head.w1, w2=wl.head.w2)
        kw = dict(kw, H=wl.H[t])
    return w, kw


def run_oracle(wl, t=0, **kw):
    w, kw = _oracle_inputs(wl, t, kw)
    return oracle.build_tree(wl.logits[t], wl.weights.emb, wl.weights.dtype, w,
                             None if wl.h0 is None else wl.h0[t], wl.M, wl.B, wl.T,
                             logits_dtype=wl.logits_dtype, **kw)


def rescore(wl, t, tokens, parents, n, **kw):
    w, kw = _oracle_inputs(wl, t, kw)
    return oracle.score_paths(wl.logits[t], wl.weights.emb, wl.weights.dtype, w,
                              None if wl.h0 is None else wl.h0[t], wl.M, wl.B, wl.T,
                              tokens, parents, n, logits_dtype=wl.logits_dtype, **kw)


def check_tree_valid(tok, par, dep, pos, mask, scores, n, B, pos_offset=0):
    """Structural validity of an emitted tree (pop order, prefix closure, mask)."""
    errs = []
    for i in range(n):
        p = int(par[i])
        if p >= i:
            errs.append(f"node {i}: parent {p} not earlier")
            continue
        want_d = 1 if p < 0 else int(dep[p]) + 1
        if int(dep[i]) != want_d:
            errs.append(f"node {i}: depth {dep[i]} != {want_d}")
        if int(pos[i]) != pos_offset + int(dep[i]):
            errs.append(f"node {i}: position {pos[i]}")
        row = np.zeros(B, np.uint8)
        row[i] = 1
        if p >= 0:
            row |= mask[p]
            if scores[i] > scores[p]:
                errs.append(f"node {i}: score above parent")
        if not np.array_equal(mask[i], row):
            errs.append(f"node {i}: mask row")
        if i > 0 and scores[i] > scores[i - 1]:
            errs.append(f"node {i}: pop order not monotone")
    for i in range(n, B):
        if tok[i] != -1 or par[i] != -1 or dep[i] != 0 or mask[i].any() or scores[i] != -math.inf:
            errs.append(f"pad row {i}")
    return errs

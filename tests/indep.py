"""Independent cross-checkers that pin the oracle (CPU only, small shapes).

None of this imports the oracle.  The scorer below takes a different route to
the same quantities: it applies the correction over the *full* vocabulary with
the out-of-slice entries masked back to the base logits, normalises with
torch.log_softmax, and advances the state with torch.nn.GRUCell.  Under the
TAIL reading the two definitions coincide exactly.
"""
from __future__ import annotations

import heapq
import itertools
import math
from typing import Dict, List, Optional, Tuple

import numpy as np
import torch


def _f64(a, dtype):
    if a is None:
        return None
    if dtype == 1:  # bf16 bits
        u = np.asarray(a, np.uint16).astype(np.uint32) << np.uint32(16)
        return torch.from_numpy(u.view(np.float32).astype(np.float64))
    return torch.from_numpy(np.asarray(a, np.float32).astype(np.float64))


class TorchScorer:
    """Full-vocabulary Domino scorer for one tree (Fact B, section 2.3)."""

    def __init__(self, X, logits_dtype, w, h0, M, T, norm_slice=False):
        self.X = _f64(X, logits_dtype)                    # [L, V]
        self.L, self.V = self.X.shape
        self.E = _f64(w.emb, w.dtype)
        d_in, d_h = self.E.shape[1], w.w_hh.shape[1]
        self.cell = torch.nn.GRUCell(d_in, d_h, bias=w.b_ih is not None).double()
        with torch.no_grad():
            self.cell.weight_ih.copy_(_f64(w.w_ih, w.dtype))
            self.cell.weight_hh.copy_(_f64(w.w_hh, w.dtype))
            if w.b_ih is not None:
                self.cell.bias_ih.copy_(_f64(w.b_ih, w.dtype))
                self.cell.bias_hh.copy_(_f64(w.b_hh, w.dtype))
        self.Wc = _f64(w.w_c, w.dtype)
        self.bc = _f64(w.b_c, w.dtype)
        self.h0 = torch.zeros(d_h, dtype=torch.float64) if h0 is None else torch.as_tensor(
            np.asarray(h0, np.float64))
        self.M = M
        self.tau = T if T > 0 else 1.0
        self.norm_slice = norm_slice
        # slices: plain python sort on (value desc, id asc)
        self.slices = []
        for d in range(self.L):
            row = self.X[d].tolist()
            self.slices.append(sorted(range(self.V), key=lambda v: (-row[v], v))[:M])

    def step(self, S, token):
        with torch.no_grad():
            return self.cell(self.E[token][None], S[None])[0]

    def logprobs(self, S, d) -> Dict[int, float]:
        """token -> corrected log-prob at depth d (only slice tokens, live only)."""
        with torch.no_grad():
            q = torch.nn.functional.linear(S, self.Wc, self.bc)
            delta = self.E @ q                                   # [V] full vocabulary
            sl = torch.tensor(self.slices[d - 1])
            y = self.X[d - 1].clone()
            y[sl] = y[sl] + delta[sl]
            if self.norm_slice:
                lp = torch.log_softmax(y[sl] / self.tau, dim=0)
                out = {int(t): float(v) for t, v in zip(sl.tolist(), lp.tolist())}
            else:
                lp = torch.log_softmax(y / self.tau, dim=0)
                out = {int(t): float(lp[t]) for t in sl.tolist()}
        return {t: v for t, v in out.items() if self.X[d - 1, t] > -math.inf}

    def ranked_children(self, S, d, k) -> List[Tuple[int, float]]:
        lp = self.logprobs(S, d)
        slot = {t: i for i, t in enumerate(self.slices[d - 1])}
        kids = sorted(lp.items(), key=lambda kv: (-kv[1], slot[kv[0]]))
        return kids[:k]


def enumerate_paths(sc: TorchScorer, k: int):
    """Every node of the k-restricted candidate tree: {path tuple: g}."""
    out = {}

    def rec(path, S, g, d):
        for tok, ell in sc.ranked_children(S, d, k):
            p = path + (tok,)
            out[p] = g + ell
            if d < sc.L:
                rec(p, sc.step(S, tok), g + ell, d + 1)

    rec((), sc.h0, 0.0, 1)
    return out


def top_b_paths(paths: Dict[tuple, float], B: int):
    """Top-B set by g; returns (set, gap between the B-th and (B+1)-th score)."""
    items = sorted(paths.items(), key=lambda kv: -kv[1])
    top = items[:B]
    gap = math.inf if len(items) <= B else top[-1][1] - items[B][1]
    return {p for p, _ in top}, gap


def tree_paths(tokens, parents, n) -> List[tuple]:
    paths = []
    for i in range(n):
        p = int(parents[i])
        paths.append((paths[p] if p >= 0 else ()) + (int(tokens[i]),))
    return paths


def factorized_tree(X, logits_dtype, M, B, T, k, norm_slice=False):
    """DDTree's heap over per-depth marginal menus (section 2.4, Marg children).

    Returns pop-order (tokens, parents, depth, g).
    """
    Xt = _f64(X, logits_dtype)
    L, V = Xt.shape
    tau = T if T > 0 else 1.0
    menus = []
    for d in range(L):
        row = Xt[d].tolist()
        sl = sorted(range(V), key=lambda v: (-row[v], v))[:M]
        if norm_slice:
            lp = torch.log_softmax(Xt[d, sl] / tau, dim=0).tolist()
        else:
            full = torch.log_softmax(Xt[d] / tau, dim=0)
            lp = [float(full[t]) for t in sl]
        menu = [(t, l, i) for i, (t, l) in enumerate(zip(sl, lp)) if row[t] > -math.inf]
        menu.sort(key=lambda e: (-e[1], e[2]))
        menus.append(menu[:k])
    heap, cnt = [], itertools.count()
    for t, l, _ in menus[0]:
        heapq.heappush(heap, (-l, next(cnt), t, l, 1, -1))
    toks, pars, deps, gs = [], [], [], []
    while len(toks) < B and heap:
        _, _, t, g, d, p = heapq.heappop(heap)
        i = len(toks)
        toks.append(t), pars.append(p), deps.append(d), gs.append(g)
        if d < L:
            for ct, cl, _ in menus[d]:
                heapq.heappush(heap, (-(g + cl), next(cnt), ct, g + cl, d + 1, i))
    return toks, pars, deps, gs


def _menu_heap(menus, B: int, L: int):
    """DDTree's heap over per-depth menus of (token, log-prob) in rank order."""
    heap, cnt = [], itertools.count()
    for t, l in menus[0]:
        heapq.heappush(heap, (-l, next(cnt), t, l, 1, -1))
    toks, pars, deps, gs = [], [], [], []
    while len(toks) < B and heap:
        _, _, t, g, d, p = heapq.heappop(heap)
        i = len(toks)
        toks.append(t), pars.append(p), deps.append(d), gs.append(g)
        if d < L:
            for ct, cl in menus[d]:
                heapq.heappush(heap, (-(g + cl), next(cnt), ct, g + cl, d + 1, i))
    return toks, pars, deps, gs


def static_tree(sc: TorchScorer, B: int, k: int):
    """Cond-static arm (Appendix D): the corrected menu of depth d is computed once,
    from the state of Domino's greedy chain (the best corrected child at every
    depth), and offered to every node of depth d.  Returns pop-order
    (tokens, parents, depth, g)."""
    S, menus = sc.h0, []
    for d in range(1, sc.L + 1):
        kids = sc.ranked_children(S, d, sc.M) if S is not None else []
        menus.append(kids[:k])
        S = sc.step(S, kids[0][0]) if kids else None
    return _menu_heap(menus, B, sc.L)


def greedy_chain(sc: TorchScorer, length: int):
    """Domino's chain decoder at T=0 (Fact A): argmax of the corrected logits."""
    S, toks = sc.h0, []
    for d in range(1, length + 1):
        with torch.no_grad():
            q = torch.nn.functional.linear(S, sc.Wc, sc.bc)
            sl = sc.slices[d - 1]
            zs = [(float(sc.X[d - 1, t] + sc.E[t] @ q), -i, t) for i, t in enumerate(sl)
                  if sc.X[d - 1, t] > -math.inf]
        _, _, tok = max(zs)
        toks.append(tok)
        S = sc.step(S, tok)
    return toks


def frontier_tree(sc: TorchScorer, B: int, k: int, W: Optional[int] = None):
    """Depth-synchronous frontier builder with a ledger and global top-B (Appendix B).

    Returns the selected node set as paths (W = B recovers the heap's tree).
    """
    W = B if W is None else W
    ledger = {}                      # path -> g
    frontier = [((), sc.h0, 0.0)]
    for d in range(1, sc.L + 1):
        scored = []
        for path, S, g in frontier:
            for tok, ell in sc.ranked_children(S, d, k):
                scored.append((g + ell, path + (tok,), S, tok))
        for g, p, _, _ in scored:
            ledger[p] = g
        scored.sort(key=lambda e: -e[0])
        keep = scored[:W]
        frontier = [(p, sc.step(S, tok), g) for g, p, S, tok in keep]
        if not frontier:
            break
    items = sorted(ledger.items(), key=lambda kv: -kv[1])[:B]
    return {p for p, _ in items}


class HeadTorchScorer(TorchScorer):
    """The same full-vocabulary scorer with Domino's own head (section 2.3):
    delta = W_2 SiLU(W_1 [H_d; S]) over every token, torch.nn.functional.silu."""

    def __init__(self, X, logits_dtype, w, head, H, h0, M, T, norm_slice=False):
        super().__init__(X, logits_dtype, w, h0, M, T, norm_slice)
        self.W1 = _f64(head.w1, head.dtype)
        self.W2 = _f64(head.w2, head.dtype)
        self.H = _f64(H, head.dtype)

    def logprobs(self, S, d) -> Dict[int, float]:
        with torch.no_grad():
            hs = torch.cat([self.H[d - 1], S])
            delta = self.W2 @ torch.nn.functional.silu(torch.nn.functional.linear(hs, self.W1))
            sl = torch.tensor(self.slices[d - 1])
            y = self.X[d - 1].clone()
            y[sl] = y[sl] + delta[sl]
            if self.norm_slice:
                lp = torch.log_softmax(y[sl] / self.tau, dim=0)
                out = {int(t): float(v) for t, v in zip(sl.tolist(), lp.tolist())}
            else:
                lp = torch.log_softmax(y / self.tau, dim=0)
                out = {int(t): float(lp[t]) for t in sl.tolist()}
        return {t: v for t, v in out.items() if self.X[d - 1, t] > -math.inf}


def menu_tree(sc: TorchScorer, B: int, k: int, S):
    """DDTree's heap when every node of depth d is offered the same menu, the
    top-k children of state S at that depth (a path-independent scorer)."""
    menus = [sc.ranked_children(S, d, k) for d in range(1, sc.L + 1)]
    return _menu_heap(menus, B, sc.L)

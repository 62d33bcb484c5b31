"""Oracle: a plain, slow CPU implementation of the DominoTree draft-tree builder.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call
this module; only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code with the HIP library.

Everything is computed in float64 from the exact stored input values (bf16
and fp32 widen to float64 exactly).  The code follows the paper's text in its
own order:

* Domino's causal encoder is a single-layer GRU over the embeddings of the
  tokens realised along the path (section 2.3); the gate equations are the
  PyTorch GRUCell ones (gates r, z, n) because the paper does not print them.
* The correction is the linear head q = W_c S + b_c dotted with the candidate
  embedding rows, delta(v) = E[v] . q, restricted to the depth's top-M slice
  (section 3.2, candidate restriction).
* Children(S, d) scores the slice with the corrected logits, normalises them,
  keeps the top-k and advances the GRU once per kept child (Alg. 1, step 2).
* The tree is grown by a max-heap keyed by cumulative log-probability, popped
  until the budget is spent (Alg. 1, steps 3-4; DDTree heap, section 2.4).
* Emission orders nodes so parents precede children and builds the
  ancestor-only verification mask (section 3.5; Appendix B, frontier selection).
* The ablation arms' children functions (Appendix D, the three arms; Marg
  children, section 3.1): MARG scores a depth's slice from the marginal logits
  alone (no correction; one menu per depth, shared by all its nodes);
  STATIC applies the correction once per depth, from the state of the greedy
  chain (Domino's own decoder: at each depth the best corrected child), and
  shares that corrected menu with every node of the depth.
* HEAD is Domino's own correction head (section 2.3): a rank-r bottleneck
  over the concatenation of the drafter's hidden state at the position and
  the path state, delta = W_2 SiLU(W_1 [H_d; S]), with W_2's rows gathered
  for the depth's slice.  The paper prints no biases, so there are none.
* The adaptive budget (CaDDTree's stopping rule, section 2.5, carried into
  the conditional pop loop, section 3.4): with the cost model (C_d, C_v(n))
  given, the loop keeps Phi(n) = sum of pi_s = exp(g_s) over the nodes popped
  so far and stops the first time theta(n) = (1 + Phi(n)) / (C_d + C_v(n))
  does not improve on theta(n - 1); that node is not kept.  B is the cap.
* The frontier builder (Appendix B, frontier ledger and selection; section
  4.5.1, batched construction for serving): W lanes advance depth by depth;
  every child a lane scores goes into a ledger; the top W of each depth
  become the next lanes; the tree is the ledger's global top B.  With W >= B
  it selects the heap's node set.

Readings of the paper that this file fixes (the paper is silent on them):

* Normalisation (TAIL, default): logZ = LSE(corrected slice logits, R_d) where
  R_d is the log-sum-exp of the *uncorrected* logits outside the slice, so a
  zeroed correction gives exactly the full-vocabulary marginal log-probs.
  SLICE normalises over the slice only.
* Temperature: tau = T if T > 0 else 1; logits are divided by tau before the
  log-softmax; the top-M selection uses the raw logits.
* Ties: top-M by (logit desc, token id asc); children by (log-prob desc,
  slot asc); heap by (g desc, insertion id asc), children inserted in rank order.
* HEAD: no biases in either layer; W_1's columns are [H_d; S] in that order;
  H's row d-1 scores depth d, like the logits' row d-1.
* k (children per expansion) = min(M, B) unless max_children > 0, then
  min(max_children, M).
* Dead slots (logit == -inf) are never returned as children.  A tree whose
  logits hold NaN or +inf gets status NONFINITE and no nodes.
* Padding rows: token -1, parent -1, depth 0, position pos_offset,
  score -inf, all-zero mask row.
* Frontier builder: lanes keep ledger order (a lane's children follow the
  children of the lanes before it); the top W of a depth are taken by
  (g desc, ledger order); the final top B by (g desc, depth asc, ledger order)
  -- the depth-then-lane tie rule -- and the tree is emitted in that order
  (parents first: a child never scores above its parent).  D = L depths.
* Adaptive budget: pi_s is the node's cumulative path probability exp(g_s)
  (the paper sums the heap's cumulative path log-probs); "stops improving"
  is theta(n) <= theta(n-1); the tree may stop at 0 nodes; theta(0) uses
  C_v(0); the cost model is an input (the paper gives none).

Pins: see tests/test_oracle_*.py (library routines, brute force, closed forms,
the greedy chain, the factorised tree, a frontier builder, a hand-derived
golden tree).  Absolute score values at the full workload sizes beyond those
pins are "parity unpinned": the paper prints no worked example.
"""
from __future__ import annotations

import heapq
import math
from typing import List, Optional, Sequence

import numpy as np

NORM_TAIL = 0
NORM_SLICE = 1
SCORER_COND = 0    # DominoTree: the correction recomputed from each node's own path state
SCORER_MARG = 1    # Marg: marginal logits only
SCORER_STATIC = 2  # Cond-static: the correction along the greedy chain, one menu per depth
SCORER_HEAD = 3    # Domino's rank-r SiLU head over [H_d; S], recomputed per node
TREE_NONFINITE = 0x1

DT_F32 = 0
DT_BF16 = 1


# ---------------------------------------------------------------------------
# input decoding
# ---------------------------------------------------------------------------

def widen(a: np.ndarray, dtype: int) -> np.ndarray:
    """Stored tensor -> float64.  bf16 arrives as uint16 bit patterns."""
    if a is None:
        return None
    if dtype == DT_BF16:
        u = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def effective_temperature(T: float) -> float:
    """tau = T for T > 0; T = 0 (deterministic drafting) scores with tau = 1."""
    return float(T) if T > 0 else 1.0


def logsumexp(a: np.ndarray) -> float:
    """log sum exp of a 1-D float64 array; -inf for an empty or all -inf array."""
    if a.size == 0:
        return -math.inf
    m = float(np.max(a))
    if m == -math.inf:
        return -math.inf
    return m + math.log(float(np.sum(np.exp(a - m))))


# ---------------------------------------------------------------------------
# Alg. 1 step 1: per-depth marginal top-M (candidate restriction, section 3.2)
# ---------------------------------------------------------------------------

def scan_row(x: np.ndarray, M: int, tau: float):
    """Top-M token ids of one depth's marginal logits and the tail log-sum-exp.

    Returns (ids[M] int64 ordered by (logit desc, id asc), logits[M] float64,
    R) where R = log sum_{v not in ids} exp(x[v] / tau) (-inf if empty).
    """
    x = np.asarray(x, dtype=np.float64)
    order = np.argsort(-x, kind="stable")      # stable: equal logits keep id order
    ids = order[:M].astype(np.int64)
    tail = np.ones(x.shape[0], dtype=bool)
    tail[ids] = False
    R = logsumexp(x[tail] / tau)
    return ids, x[ids], R


# ---------------------------------------------------------------------------
# Domino's causal encoder (section 2.3), PyTorch GRUCell convention
# ---------------------------------------------------------------------------

def sigmoid(a: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-a))


def silu(a: np.ndarray) -> np.ndarray:
    """SiLU(a) = a * sigmoid(a), the head's nonlinearity (section 2.3)."""
    return a * sigmoid(a)


def gru_cell(h: np.ndarray, xs: np.ndarray, w_ih, w_hh, b_ih, b_hh) -> np.ndarray:
    """Advance state h [d_h] by each input row of xs [k, d_in]; returns [k, d_h].

    r = sigmoid(W_ir x + b_ir + W_hr h + b_hr)
    z = sigmoid(W_iz x + b_iz + W_hz h + b_hz)
    n = tanh(W_in x + b_in + r * (W_hn h + b_hn))
    h' = (1 - z) * n + z * h
    """
    d_h = h.shape[0]
    gi = xs @ w_ih.T                      # [k, 3 d_h]
    if b_ih is not None:
        gi = gi + b_ih
    gh = w_hh @ h                         # [3 d_h]
    if b_hh is not None:
        gh = gh + b_hh
    i_r, i_z, i_n = gi[:, :d_h], gi[:, d_h:2 * d_h], gi[:, 2 * d_h:]
    h_r, h_z, h_n = gh[:d_h], gh[d_h:2 * d_h], gh[2 * d_h:]
    r = sigmoid(i_r + h_r)
    z = sigmoid(i_z + h_z)
    n = np.tanh(i_n + r * h_n)
    return (1.0 - z) * n + z * h


# ---------------------------------------------------------------------------
# the builder
# ---------------------------------------------------------------------------

class _Model:
    """float64 copies of the weights plus the per-depth candidate tables."""

    def __init__(self, X, emb, emb_dtype, w, M, tau, norm_mode, scorer=SCORER_COND, H=None):
        self.L = X.shape[0]
        self.M = M
        self.tau = tau
        self.norm_mode = norm_mode
        self.scorer = scorer
        self.menus = None
        self.w_ih = widen(w["w_ih"], w["dtype"])
        self.w_hh = widen(w["w_hh"], w["dtype"])
        self.b_ih = widen(w.get("b_ih"), w["dtype"])
        self.b_hh = widen(w.get("b_hh"), w["dtype"])
        self.w_c = widen(w["w_c"], w["dtype"])
        self.b_c = widen(w.get("b_c"), w["dtype"])
        # Alg. 1 step 1, once per depth: top-M ids, their logits, their embeddings
        self.cand, self.xc, self.R, self.Ec = [], [], [], []
        for d in range(self.L):
            ids, xs, R = scan_row(X[d], M, tau)
            self.cand.append(ids)
            self.xc.append(xs)
            self.R.append(R)
            self.Ec.append(widen(np.asarray(emb)[ids], emb_dtype))
        if scorer == SCORER_HEAD:
            # section 2.3: W_1 acts on [H_d; S]; its H half is path-independent,
            # so a_d = W_1^H H_d once per depth; W_2's rows for the slice
            w1 = widen(w["w1"], w["dtype"])
            d_H = w1.shape[1] - self.w_hh.shape[1]
            Hd = widen(H, w["dtype"])
            self.w1s = w1[:, d_H:]
            self.a = [w1[:, :d_H] @ Hd[d] for d in range(self.L)]
            self.W2c = [widen(np.asarray(w["w2"])[ids], w["dtype"]) for ids in self.cand]

    def slot_logprobs(self, S: Optional[np.ndarray], d: int):
        """Corrected, normalised log-probs of depth d's slice given path state S.

        delta_m = E[cand_d[m]] . (W_c S + b_c) (HEAD: W_2[cand_d[m]] .
        SiLU(a_d + W_1^S S));  z = (x + delta) / tau;  ell = z - logZ.
        S = None: no correction (delta = 0, the marginals).
        Returns (ell[M] with -inf for dead slots, live mask).
        """
        if S is None:
            delta = np.zeros(self.M)
        elif self.scorer == SCORER_HEAD:
            y = silu(self.a[d - 1] + self.w1s @ S)
            delta = self.W2c[d - 1] @ y
        else:
            q = self.w_c @ S
            if self.b_c is not None:
                q = q + self.b_c
            delta = self.Ec[d - 1] @ q
        x = self.xc[d - 1]
        live = x > -math.inf
        z = np.full(self.M, -math.inf)
        z[live] = (x[live] + delta[live]) / self.tau
        if self.norm_mode == NORM_SLICE:
            logZ = logsumexp(z[live])
        else:
            logZ = logsumexp(np.append(z[live], self.R[d - 1]))
        ell = np.full(self.M, -math.inf)
        ell[live] = z[live] - logZ
        return ell, live

    def static_menus(self, S0: np.ndarray):
        """Cond-static menus: walk the greedy chain from S0 (at each depth the best
        corrected slot, by (ell desc, slot asc)), keeping every depth's corrected,
        normalised slice log-probs.  Depths past a dead end get no live slot."""
        self.menus = []
        S = S0
        for d in range(1, self.L + 1):
            if S is None:
                self.menus.append((np.full(self.M, -math.inf), np.zeros(self.M, bool)))
                continue
            ell, live = self.slot_logprobs(S, d)
            self.menus.append((ell, live))
            slots = [m for m in range(self.M) if live[m]]
            if not slots:
                S = None
                continue
            best = min(slots, key=lambda m: (-ell[m], m))
            S = gru_cell(S, self.Ec[d - 1][[best]], self.w_ih, self.w_hh, self.b_ih, self.b_hh)[0]

    def menu(self, S: Optional[np.ndarray], d: int):
        """The log-probs the children function ranks at depth d (all M slots)."""
        if self.scorer == SCORER_MARG:
            return self.slot_logprobs(None, d)
        if self.scorer == SCORER_STATIC:
            return self.menus[d - 1]
        return self.slot_logprobs(S, d)

    def children(self, S: Optional[np.ndarray], d: int, k: int, gaps: list):
        """Children(S_{d-1}, d) of Alg. 1 step 2: top-k (token, ell, slot, child state).

        Returns (children, ell_out) where ell_out is the log-prob of the best
        slot left out by the top-k cut (-inf if none).  The gap between the k-th
        and (k+1)-th log-prob is logged as a "children" gap.  MARG and STATIC
        ignore S (their menus are path-independent) and return no child states."""
        ell, live = self.menu(S, d)
        slots = [m for m in range(self.M) if live[m]]
        slots.sort(key=lambda m: (-ell[m], m))
        ell_out = -math.inf
        if len(slots) > k:
            ell_out = float(ell[slots[k]])
            gaps.append(("children", ell[slots[k - 1]] - ell[slots[k]]))
        kept = slots[:k]
        if not kept:
            return [], ell_out
        tokens = [int(self.cand[d - 1][m]) for m in kept]
        if self.scorer not in (SCORER_COND, SCORER_HEAD):
            return [(tokens[i], float(ell[m]), m, None) for i, m in enumerate(kept)], ell_out
        states = gru_cell(S, self.Ec[d - 1][kept], self.w_ih, self.w_hh, self.b_ih, self.b_hh)
        return [(tokens[i], float(ell[m]), m, states[i]) for i, m in enumerate(kept)], ell_out


def _empty_tree(B: int, pos_offset: int, status: int):
    return {
        "tokens": np.full(B, -1, np.int32),
        "parents": np.full(B, -1, np.int32),
        "depth": np.zeros(B, np.int32),
        "position_ids": np.full(B, pos_offset, np.int32),
        "mask": np.zeros((B, B), np.uint8),
        "scores": np.full(B, -np.inf, np.float64),
        "slots": np.full(B, -1, np.int32),
        "ell": np.full(B, -np.inf, np.float64),
        "ell_out": np.full(B, -np.inf, np.float64),
        "rank": np.full(B, -1, np.int32),
        "n_nodes": 0,
        "status": status,
        "min_gap": math.inf,
        "gaps": [],
        "excluded": -math.inf,
    }


def build_tree(X: np.ndarray, emb: np.ndarray, emb_dtype: int, weights: dict,
               h0: Optional[np.ndarray], M: int, B: int, T: float,
               max_children: int = 0, norm_mode: int = NORM_TAIL, pos_offset: int = 0,
               logits_dtype: int = DT_F32, scorer: int = SCORER_COND, H: Optional[np.ndarray] = None,
               budget_costs=None, frontier_width: int = 0):
    """Build one draft tree (Alg. 1) and emit it in pop order.

    X: [L, V] stored marginal logits of one tree; emb: [V, d_e]; weights: dict
    with w_ih, w_hh, b_ih, b_hh, w_c, b_c, dtype (HEAD: also w1 [r, d_H + d_h]
    and w2 [V, r]); h0: [d_h] or None (zeros); H: [L, d_H], HEAD only.
    budget_costs: None (fixed budget B) or (C_d, C_v[0..B]) for the adaptive
    budget, B then being the cap.
    frontier_width: 0 (the heap of Alg. 1) or W >= 1 (the frontier builder of
    Appendix B with W lanes; not combined with budget_costs).
    Returns a dict of emitted arrays plus the smallest decisive score gap.
    """
    Xd = widen(X, logits_dtype)
    if np.any(np.isnan(Xd)) or np.any(Xd == math.inf):
        return _empty_tree(B, pos_offset, TREE_NONFINITE)
    tau = effective_temperature(T)
    k = min(M, B) if max_children <= 0 else min(max_children, M)
    model = _Model(Xd, emb, emb_dtype, weights, M, tau, norm_mode, scorer, H)
    L = model.L
    d_h = model.w_hh.shape[1]
    S0 = np.zeros(d_h) if h0 is None else np.asarray(h0, np.float64)
    if scorer == SCORER_STATIC:
        model.static_menus(S0)
    if frontier_width > 0:
        if budget_costs is not None:
            raise ValueError("the adaptive budget applies to the heap builder only")
        return _frontier_tree(model, S0, k, B, frontier_width, pos_offset)

    gaps: list = []    # (kind, value): the decisive score gaps
    heap = []          # entries (-g, insertion id, payload)
    next_id = 0
    # Alg. 1 step 3: the root's children
    kids, ell_out = model.children(S0, 1, k, gaps)
    for r, (tok, ell, m, S) in enumerate(kids):
        heapq.heappush(heap, (-ell, next_id, (tok, ell, m, S, 1, -1, ell, ell_out, r)))
        next_id += 1
    # Alg. 1 step 4: pop the best entry, add it to the tree, push its children
    tree = []          # (token, g, slot, depth, parent pop index, ell, ell_out, rank)
    if budget_costs is not None:
        c_d, c_v = float(budget_costs[0]), np.asarray(budget_costs[1], np.float64)
        phi = 0.0
        theta = 1.0 / (c_d + c_v[0])   # theta(0): the empty tree
    while len(tree) < B and heap:
        if budget_costs is not None:
            # adaptive budget: theta(n) with the best entry as node n
            n = len(tree) + 1
            th = (1.0 + phi + math.exp(-heap[0][0])) / (c_d + c_v[n])
            gaps.append(("budget", abs(th - theta) / theta))
            if th <= theta:
                break            # theta stops improving: node n is not kept
            phi += math.exp(-heap[0][0])
            theta = th
        neg_g, _, (tok, g, m, S, d, parent, ell, eo, r) = heapq.heappop(heap)
        i = len(tree)
        tree.append((tok, g, m, d, parent, ell, eo, r))
        if d < L:
            kids, ell_out = model.children(S, d + 1, k, gaps)
            for rr, (ctok, cell, cm, cS) in enumerate(kids):
                heapq.heappush(heap, (-(g + cell), next_id,
                                      (ctok, g + cell, cm, cS, d + 1, i, cell, ell_out, rr)))
                next_id += 1
    # decisive gaps: consecutive pops and the last pop vs the best entry left out
    for i in range(len(tree) - 1):
        gaps.append(("pop", tree[i][1] - tree[i + 1][1]))
    excluded = -math.inf
    if heap:
        excluded = -heap[0][0]
        if len(tree) == B or (budget_costs is not None and tree):
            gaps.append(("boundary", tree[-1][1] - excluded))
    out = _emit(tree, B, pos_offset, min(v for _, v in gaps) if gaps else math.inf)
    out["gaps"] = gaps
    out["excluded"] = excluded
    return out


def _frontier_tree(model, S0, k: int, B: int, W: int, pos_offset: int):
    """The frontier builder (Appendix B): W lanes per depth, a ledger of every
    scored child, the global top B of the ledger."""
    gaps: list = []
    # ledger entries: [g, depth, token, parent ledger index, ell, ell_out, rank, slot]
    ledger = []
    lanes = [(-1, S0, 0.0)]        # (ledger index of the lane's node, path state, g)
    cuts = []                      # (depth, W-th minus (W+1)-th score of the depth)
    for d in range(1, model.L + 1):
        row = []                   # ledger indices scored at this depth, in ledger order
        states = {}
        for li, S, g in lanes:
            kids, ell_out = model.children(S, d, k, gaps)
            for r, (tok, ell, m, cS) in enumerate(kids):
                row.append(len(ledger))
                states[len(ledger)] = cS
                ledger.append([g + ell, d, tok, li, ell, ell_out, r, m])
        if not row or d == model.L:
            break
        # the top W of this depth by (g desc, ledger order) advance, in ledger order
        best = sorted(row, key=lambda e: (-ledger[e][0], e))
        if len(best) > W:
            gaps.append(("frontier", ledger[best[W - 1]][0] - ledger[best[W]][0]))
            cuts.append((d, ledger[best[W - 1]][0] - ledger[best[W]][0]))
        keep = sorted(best[:W])
        lanes = [(e, states[e], ledger[e][0]) for e in keep]
    # the tree: the ledger's global top B by (g desc, depth asc, ledger order)
    order = sorted(range(len(ledger)), key=lambda e: (-ledger[e][0], ledger[e][1], e))
    sel = order[:B]
    pos = {e: i for i, e in enumerate(sel)}
    tree = []
    for e in sel:
        g, d, tok, li, ell, eo, r, m = ledger[e]
        tree.append((tok, g, m, d, -1 if li < 0 else pos[li], ell, eo, r))
    for i in range(len(tree) - 1):
        gaps.append(("pop", tree[i][1] - tree[i + 1][1]))
    excluded = ledger[order[B]][0] if len(order) > B else -math.inf
    if len(order) > B:
        gaps.append(("boundary", tree[-1][1] - excluded))
    out = _emit(tree, B, pos_offset, min(v for _, v in gaps) if gaps else math.inf)
    out["gaps"] = gaps
    out["excluded"] = excluded
    out["frontier_cut"] = cuts
    return out


def _emit(tree, B: int, pos_offset: int, min_gap: float):
    """Pop-order arrays and the ancestor-or-self mask (section 3.5)."""
    out = _empty_tree(B, pos_offset, 0)
    n = len(tree)
    for i, (tok, g, m, d, parent, ell, ell_out, rank) in enumerate(tree):
        out["ell"][i] = ell
        out["ell_out"][i] = ell_out
        out["rank"][i] = rank
        out["tokens"][i] = tok
        out["parents"][i] = parent
        out["depth"][i] = d
        out["position_ids"][i] = pos_offset + d
        out["scores"][i] = g
        out["slots"][i] = m
        out["mask"][i, i] = 1
        if parent >= 0:
            out["mask"][i] |= out["mask"][parent]
    out["n_nodes"] = n
    out["min_gap"] = min_gap
    return out


def build_trees(logits: np.ndarray, logits_dtype: int, emb: np.ndarray, emb_dtype: int,
                weights: dict, h0: Optional[np.ndarray], M: int, B: int, T: float,
                max_children: int = 0, norm_mode: int = NORM_TAIL, pos_offset: int = 0,
                trees: Optional[Sequence[int]] = None, scorer: int = SCORER_COND,
                H: Optional[np.ndarray] = None, budget_costs=None, frontier_width: int = 0):
    """build_tree over the batch (or the listed tree indices); H: [b, L, d_H]."""
    idx = range(logits.shape[0]) if trees is None else trees
    return [build_tree(logits[t], emb, emb_dtype, weights, None if h0 is None else h0[t],
                       M, B, T, max_children, norm_mode, pos_offset, logits_dtype, scorer,
                       None if H is None else H[t], budget_costs, frontier_width)
            for t in idx]


def scan(logits: np.ndarray, logits_dtype: int, M: int, T: float):
    """Alg. 1 step 1 for every row of a [rows, V] array: (ids, logits, R)."""
    X = widen(logits, logits_dtype)
    tau = effective_temperature(T)
    ids = np.zeros((X.shape[0], M), np.int64)
    xs = np.zeros((X.shape[0], M))
    R = np.zeros(X.shape[0])
    for r in range(X.shape[0]):
        ids[r], xs[r], R[r] = scan_row(X[r], M, tau)
    return ids, xs, R


def score_paths(X: np.ndarray, emb: np.ndarray, emb_dtype: int, weights: dict,
                h0: Optional[np.ndarray], M: int, B: int, T: float, tokens, parents, n_nodes: int,
                max_children: int = 0, norm_mode: int = NORM_TAIL, logits_dtype: int = DT_F32,
                scorer: int = SCORER_COND, H: Optional[np.ndarray] = None, tie_tol: float = 0.0):
    """Re-score a given tree with the oracle's Children function.

    Returns (g[n], valid): g[i] is the cumulative log-prob of node i along its
    own path; valid is False when a parent index is not earlier, a node lies
    below depth L, or a node is not among the top-k children of its parent's
    path.  With tie_tol = 0 the top-k is the exact (log-prob desc, slot asc)
    cut; with tie_tol > 0 a node also counts as a top-k child when fewer than k
    live slots beat its log-prob by more than tie_tol (a child whose log-prob is
    that close to the cut may take the k-th place).
    """
    Xd = widen(X, logits_dtype)
    tau = effective_temperature(T)
    k = min(M, B) if max_children <= 0 else min(max_children, M)
    model = _Model(Xd, emb, emb_dtype, weights, M, tau, norm_mode, scorer, H)
    d_h = model.w_hh.shape[1]
    S0 = np.zeros(d_h) if h0 is None else np.asarray(h0, np.float64)
    if scorer == SCORER_STATIC:
        model.static_menus(S0)
    g = np.zeros(n_nodes)
    state = [None] * n_nodes
    depth = [0] * n_nodes
    for i in range(n_nodes):
        p = int(parents[i])
        if p >= i:
            return g, False
        S, gp, d = (S0, 0.0, 1) if p < 0 else (state[p], g[p], depth[p] + 1)
        if d > model.L:
            return g, False
        ell, live = model.menu(S, d)
        hit = np.flatnonzero(model.cand[d - 1] == int(tokens[i]))
        if hit.size == 0 or not live[hit[0]]:
            return g, False
        m = int(hit[0])
        if tie_tol > 0:
            above = int(np.sum(live & (ell > ell[m] + tie_tol)))
        else:
            above = int(np.sum(live & ((ell > ell[m]) | ((ell == ell[m]) & (np.arange(model.M) < m)))))
        if above >= k:
            return g, False
        g[i] = gp + ell[m]
        depth[i] = d
        if scorer in (SCORER_COND, SCORER_HEAD):
            state[i] = gru_cell(S, model.Ec[d - 1][[m]], model.w_ih, model.w_hh, model.b_ih,
                                model.b_hh)[0]
    return g, True

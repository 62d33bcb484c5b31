"""Helpers for GPU tests: upload synthetic workloads, run the library, compare with the oracle."""
from __future__ import annotations

import json
import os

import numpy as np
import torch

import oracle
import treecmp
from helpers import check_tree_valid, rescore, run_oracle
from paper_2607_08642_amd import binding, synth

GAP_TOL = treecmp.GAP_TOL   # decisive score gaps above this must give identical trees


def score_tol(wl) -> float:
    """Score tolerance: 1e-4 when everything is fp32, 2e-2 when bf16 inputs feed the correction."""
    return 1e-4 if wl.weights.dtype == synth.DT_F32 and wl.logits_dtype == synth.DT_F32 else 2e-2


def to_dev(a: np.ndarray, dtype: int, device="cuda"):
    if a is None:
        return None
    if dtype == synth.DT_BF16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


class DeviceWorkload:
    def __init__(self, wl, max_children=0, norm_mode=0, pos_offset=0, scorer=0, frontier_width=0,
                 debug_spin_limit=0):
        w = wl.weights
        self.wl = wl
        d = synth.DT_BF16 if w.dtype == synth.DT_BF16 else synth.DT_F32
        self.emb = to_dev(w.emb, d)
        self.w_ih = to_dev(w.w_ih, d)
        self.w_hh = to_dev(w.w_hh, d)
        self.b_ih = to_dev(w.b_ih, d)
        self.b_hh = to_dev(w.b_hh, d)
        self.w_c = to_dev(w.w_c, d)
        self.b_c = to_dev(w.b_c, d)
        self.logits = to_dev(wl.logits, wl.logits_dtype)
        self.h0 = None if wl.h0 is None else torch.from_numpy(wl.h0.astype(np.float32)).cuda()
        # (Domino's own head is a separate entry point of a DominoTree plan)
        pscorer = 0 if scorer == oracle.SCORER_HEAD else scorer
        self.plan = binding.Plan(self.emb, self.w_ih, self.w_hh, self.b_ih, self.b_hh, self.w_c,
                                 self.b_c, L=wl.L, M=wl.M, B=wl.B, logits_dtype=wl.logits_dtype,
                                 max_batch=wl.batch, max_children=max_children,
                                 norm_mode=norm_mode, pos_offset=pos_offset, scorer=pscorer,
                                 frontier_width=frontier_width, debug_spin_limit=debug_spin_limit)
        self.kw = dict(max_children=max_children, norm_mode=norm_mode, pos_offset=pos_offset,
                       scorer=scorer)
        if frontier_width:
            self.kw["frontier_width"] = frontier_width

    def run(self):
        if self.kw["scorer"] == oracle.SCORER_HEAD:
            hd = self.wl.head
            if not hasattr(self, "w1"):
                self.w1 = to_dev(hd.w1, hd.dtype)
                self.w2 = to_dev(hd.w2, hd.dtype)
                self.H = to_dev(self.wl.H, hd.dtype)
            tree = self.plan.build_tree_head(self.logits, self.H, self.w1, self.w2, self.wl.T,
                                             self.h0)
        else:
            tree = self.plan.build_tree(self.logits, self.wl.T, self.h0)
        torch.cuda.synchronize()
        return {k: getattr(tree, k).cpu().numpy() for k in
                ("tokens", "parents", "depth", "position_ids", "mask", "scores", "n_nodes",
                 "status")}

    def close(self):
        self.plan.close()


def compare_tree(wl, t, got, kw, tol=None, name=""):
    """Compare GPU tree t with the oracle (tie-aware: tests/treecmp.py).

    Returns (kind, max_score_err): kind 'exact' (identical node for node) or
    'banded' (identical outside near-tie bands, the bands checked as sets or by
    re-scoring); raises AssertionError on a mismatch.  With the environment
    variable PARITY_LOG set, one JSON line per tree is appended to that file."""
    tol = score_tol(wl) if tol is None else tol
    ref = run_oracle(wl, t, **kw)
    kw = {k: v for k, v in kw.items() if k not in ("budget_costs", "frontier_width")}  # (not re-scoring inputs)
    B = wl.B
    n = int(got["n_nodes"][t])
    assert int(got["status"][t]) == ref["status"], (got["status"][t], ref["status"])
    tok, par, dep = got["tokens"][t], got["parents"][t], got["depth"][t]
    pos, mask, sc = got["position_ids"][t], got["mask"][t], got["scores"][t]
    errs = check_tree_valid(tok, par, dep, pos, mask, sc, n, B, kw.get("pos_offset", 0))
    assert not errs, f"tree {t}: {errs[:5]}"
    one = {k: got[k][t] for k in ("tokens", "parents", "depth", "position_ids", "mask", "scores",
                                  "n_nodes", "status")}

    def rs(tokens, parents, nn, tie_tol):
        return rescore(wl, t, tokens, parents, nn, max_children=kw.get("max_children", 0),
                       norm_mode=kw.get("norm_mode", 0), scorer=kw.get("scorer", 0),
                       tie_tol=tie_tol)

    try:
        kind, err, n_exact = treecmp.compare(ref, one, rs, tol, GAP_TOL, B)
    except AssertionError as e:
        raise AssertionError(f"{name} tree {t}: {e}") from None
    log = os.environ.get("PARITY_LOG")
    if log:
        depth_max = int(np.max(dep[:n])) if n else 0
        with open(log, "a") as f:
            f.write(json.dumps({"case": name, "tree": t, "kind": kind, "max_score_err": err,
                                "exact_positions": n_exact, "n_nodes": n, "depth_max": depth_max,
                                "min_gap": float(ref["min_gap"])}) + "\n")
    return kind, err

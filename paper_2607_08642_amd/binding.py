"""Thin Python binding of libdominotree (include/dominotree.h).

Argument marshalling only: every step of the tree build runs in the HIP
kernels behind the C ABI.  torch is used for device memory and streams.  The
library is loaded from this package directory; if it is missing, every call
raises (there is no fallback).
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libdominotree.so")

DT_F32 = 0
DT_BF16 = 1
DT_NORM_TAIL = 0
DT_NORM_SLICE = 1
DT_SCORER_COND = 0
DT_SCORER_MARG = 1
DT_SCORER_STATIC = 2
DT_TREE_NONFINITE = 0x1
DT_TREE_TRUNCATED = 0x2
DT_TREE_TIMEOUT = 0x4
ABI_VERSION = 3

STATUS = {0: "DT_OK", -1: "DT_ERR_NULL", -2: "DT_ERR_SHAPE", -3: "DT_ERR_DTYPE",
          -4: "DT_ERR_UNSUPPORTED", -5: "DT_ERR_WORKSPACE", -6: "DT_ERR_ALIGN", -7: "DT_ERR_HIP"}

# every symbol include/dominotree.h declares
EXPORTS = ("dt_abi_version", "dt_status_string", "dt_last_error", "dt_plan_create",
           "dt_workspace_size", "dt_build_tree", "dt_plan_destroy", "dt_plan_set_profiling",
           "dt_plan_stage_ms", "dt_scan_workspace_size", "dt_scan_topm", "dt_head_workspace_size",
           "dt_build_tree_head", "dt_build_tree_noalloc",
           "dt_plan_expand_stats", "dt_plan_set_adaptive_budget", "dt_model_create",
           "dt_model_destroy", "dt_plan_create_from_model")
STAGES = ("scan", "expand")


class DTError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class dt_gru(ctypes.Structure):
    _fields_ = [("w_ih", ctypes.c_void_p), ("w_hh", ctypes.c_void_p), ("b_ih", ctypes.c_void_p),
                ("b_hh", ctypes.c_void_p), ("d_in", ctypes.c_int), ("d_h", ctypes.c_int)]


class dt_head(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p), ("b", ctypes.c_void_p)]


class dt_domino_head(ctypes.Structure):
    _fields_ = [("w1", ctypes.c_void_p), ("w2", ctypes.c_void_p), ("d_H", ctypes.c_int),
                ("rank", ctypes.c_int)]


class dt_options(ctypes.Structure):
    _fields_ = [("max_children", ctypes.c_int), ("norm_mode", ctypes.c_int),
                ("pos_offset", ctypes.c_int), ("scorer", ctypes.c_int),
                ("frontier_width", ctypes.c_int), ("debug_spin_limit", ctypes.c_int)]


class dt_tree(ctypes.Structure):
    _fields_ = [("tokens", ctypes.c_void_p), ("parents", ctypes.c_void_p),
                ("depth", ctypes.c_void_p), ("position_ids", ctypes.c_void_p),
                ("mask", ctypes.c_void_p), ("scores", ctypes.c_void_p),
                ("n_nodes", ctypes.c_void_p), ("status", ctypes.c_void_p)]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the shared library (raises if it is missing or its ABI differs)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with paper_2607_08642_amd.build.build()")
    lib = ctypes.CDLL(path)
    vp, ci, cf, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
    lib.dt_abi_version.restype = ci
    lib.dt_status_string.restype = ctypes.c_char_p
    lib.dt_status_string.argtypes = [ci]
    lib.dt_last_error.restype = ctypes.c_char_p
    lib.dt_plan_create.restype = ci
    lib.dt_plan_create.argtypes = [ctypes.POINTER(vp), vp, ci, ci, ctypes.POINTER(dt_gru),
                                   ctypes.POINTER(dt_head), ci, ci, ci, ci, ci, ci,
                                   ctypes.POINTER(dt_options)]
    lib.dt_model_create.restype = ci
    lib.dt_model_create.argtypes = [ctypes.POINTER(vp), vp, ci, ci, ctypes.POINTER(dt_gru),
                                    ctypes.POINTER(dt_head), ci]
    lib.dt_model_destroy.restype = None
    lib.dt_model_destroy.argtypes = [vp]
    lib.dt_plan_create_from_model.restype = ci
    lib.dt_plan_create_from_model.argtypes = [ctypes.POINTER(vp), vp, ci, ci, ci, ci, ci,
                                              ctypes.POINTER(dt_options)]
    lib.dt_workspace_size.restype = ci
    lib.dt_workspace_size.argtypes = [vp, ci, ctypes.POINTER(sz)]
    lib.dt_build_tree.restype = ci
    lib.dt_build_tree.argtypes = [vp, vp, ci, vp, cf, vp, sz, ctypes.POINTER(dt_tree), vp]
    lib.dt_plan_destroy.restype = None
    lib.dt_plan_destroy.argtypes = [vp]
    lib.dt_plan_set_profiling.restype = ci
    lib.dt_plan_set_profiling.argtypes = [vp, ci]
    lib.dt_plan_stage_ms.restype = ci
    lib.dt_plan_stage_ms.argtypes = [vp, ctypes.POINTER(ctypes.c_float)]
    lib.dt_scan_workspace_size.restype = ci
    lib.dt_scan_workspace_size.argtypes = [ci, ci, ci, ctypes.POINTER(sz)]
    lib.dt_scan_topm.restype = ci
    lib.dt_head_workspace_size.restype = ci
    lib.dt_head_workspace_size.argtypes = [vp, ci, ctypes.POINTER(dt_domino_head), ctypes.POINTER(sz)]
    lib.dt_build_tree_head.restype = ci
    lib.dt_build_tree_head.argtypes = [vp, vp, ci, vp, ctypes.POINTER(dt_domino_head), vp, cf, vp,
                                       sz, ctypes.POINTER(dt_tree), vp]
    lib.dt_scan_topm.argtypes = [vp, ci, ci, ci, ci, cf, vp, vp, vp, vp, vp, sz, vp]
    lib.dt_plan_set_adaptive_budget.restype = ci
    lib.dt_plan_set_adaptive_budget.argtypes = [vp, cf, ctypes.POINTER(cf), ci]
    lib.dt_plan_expand_stats.restype = ci
    lib.dt_plan_expand_stats.argtypes = [vp, vp, vp, ci]
    lib.dt_build_tree_noalloc.restype = ci
    lib.dt_build_tree_noalloc.argtypes = [vp, vp, ci, vp, cf, ctypes.POINTER(dt_tree), vp]
    if lib.dt_abi_version() != ABI_VERSION:
        raise RuntimeError(f"ABI mismatch: library {lib.dt_abi_version()} vs binding {ABI_VERSION}")
    _lib = lib
    return lib


def _check(st: int) -> None:
    if st != 0:
        raise DTError(st, load().dt_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return DT_BF16
    if t.dtype == torch.float32:
        return DT_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def _stream(stream) -> Optional[int]:
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream or None


@dataclasses.dataclass
class Tree:
    """Emitted trees (device tensors), nodes in pop order."""
    tokens: "torch.Tensor"        # [b, B] int32
    parents: "torch.Tensor"       # [b, B] int32, -1 = child of the root
    depth: "torch.Tensor"         # [b, B] int32
    position_ids: "torch.Tensor"  # [b, B] int32
    mask: "torch.Tensor"          # [b, B, B] uint8 ancestor-or-self
    scores: "torch.Tensor"        # [b, B] float32
    n_nodes: "torch.Tensor"       # [b] int32
    status: "torch.Tensor"        # [b] int32

    @staticmethod
    def empty(batch: int, B: int, device) -> "Tree":
        import torch
        i32 = dict(dtype=torch.int32, device=device)
        return Tree(torch.empty(batch, B, **i32), torch.empty(batch, B, **i32),
                    torch.empty(batch, B, **i32), torch.empty(batch, B, **i32),
                    torch.empty(batch, B, B, dtype=torch.uint8, device=device),
                    torch.empty(batch, B, dtype=torch.float32, device=device),
                    torch.empty(batch, **i32), torch.empty(batch, **i32))

    def as_c(self) -> dt_tree:
        """The dt_tree view of these tensors (built once; the tensors never move)."""
        c = self.__dict__.get("_c")
        if c is None:
            c = dt_tree(*(x.data_ptr() for x in (self.tokens, self.parents, self.depth,
                                                    self.position_ids, self.mask, self.scores,
                                                    self.n_nodes, self.status)))
            self.__dict__["_c"] = c
        return c


class Model:
    """dt_model: a drafter's vocabulary tables (embedding table folded through
    the GRU input projection and the correction head) and repacked GRU, shared
    by every Plan made from it.  The weight tensors may be freed once it exists.
    """

    def __init__(self, emb, w_ih, w_hh, b_ih, b_hh, w_c, b_c):
        lib = load()
        self._lib = lib
        self.V, self.d_e = emb.shape
        self.d_h = w_hh.shape[1]
        self.device = emb.device
        gru = dt_gru(_ptr(w_ih), _ptr(w_hh), _ptr(b_ih), _ptr(b_hh), self.d_e, self.d_h)
        head = dt_head(_ptr(w_c), _ptr(b_c))
        h = ctypes.c_void_p()
        _check(lib.dt_model_create(ctypes.byref(h), _ptr(emb), self.V, self.d_e, ctypes.byref(gru),
                                   ctypes.byref(head), _dtype_code(emb)))
        self.handle = h

    def close(self) -> None:
        """Drop this reference (the tables live on while a plan uses them)."""
        if getattr(self, "handle", None):
            self._lib.dt_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Plan:
    """dt_plan: one model (embedding table, GRU, head) and one (L, M, B) shape.

    Plan(emb, w_ih, ...) builds a model of its own (dt_plan_create);
    Plan.from_model(model, ...) shares an existing Model's tables.
    """

    def __init__(self, emb, w_ih, w_hh, b_ih, b_hh, w_c, b_c, *, L: int, M: int, B: int,
                 logits_dtype: int, max_batch: int = 1, max_children: int = 0,
                 norm_mode: int = DT_NORM_TAIL, pos_offset: int = 0,
                 scorer: int = DT_SCORER_COND, frontier_width: int = 0,
                 debug_spin_limit: int = 0):
        lib = load()
        self._lib = lib
        self.V, self.d_e = emb.shape
        self.d_h = w_hh.shape[1]
        self.device = emb.device
        self.L, self.M, self.B, self.max_batch = L, M, B, max_batch
        self.logits_dtype = logits_dtype
        wdt = _dtype_code(emb)
        gru = dt_gru(_ptr(w_ih), _ptr(w_hh), _ptr(b_ih), _ptr(b_hh), self.d_e, self.d_h)
        head = dt_head(_ptr(w_c), _ptr(b_c))
        opts = dt_options(max_children, norm_mode, pos_offset, scorer, frontier_width,
                          debug_spin_limit)
        h = ctypes.c_void_p()
        _check(lib.dt_plan_create(ctypes.byref(h), _ptr(emb), self.V, self.d_e, ctypes.byref(gru),
                                  ctypes.byref(head), wdt, L, M, B, logits_dtype, max_batch,
                                  ctypes.byref(opts)))
        self.handle = h
        self._ws = {}

    @classmethod
    def from_model(cls, model: Model, *, L: int, M: int, B: int, logits_dtype: int,
                   max_batch: int = 1, max_children: int = 0, norm_mode: int = DT_NORM_TAIL,
                   pos_offset: int = 0, scorer: int = DT_SCORER_COND, frontier_width: int = 0,
                   debug_spin_limit: int = 0) -> "Plan":
        """dt_plan_create_from_model: a plan over `model`'s tables."""
        self = cls.__new__(cls)
        self._lib = model._lib
        self.V, self.d_e, self.d_h, self.device = model.V, model.d_e, model.d_h, model.device
        self.L, self.M, self.B, self.max_batch = L, M, B, max_batch
        self.logits_dtype = logits_dtype
        opts = dt_options(max_children, norm_mode, pos_offset, scorer, frontier_width,
                          debug_spin_limit)
        h = ctypes.c_void_p()
        _check(self._lib.dt_plan_create_from_model(ctypes.byref(h), model.handle, L, M, B,
                                                   logits_dtype, max_batch, ctypes.byref(opts)))
        self.handle = h
        self._ws = {}
        return self

    def workspace_size(self, batch: int) -> int:
        n = ctypes.c_size_t()
        _check(self._lib.dt_workspace_size(self.handle, batch, ctypes.byref(n)))
        return n.value

    def workspace(self, batch: int):
        import torch
        if batch not in self._ws:
            self._ws[batch] = torch.empty(self.workspace_size(batch), dtype=torch.uint8,
                                          device=self.device)
        return self._ws[batch]

    def build_tree(self, logits, T: float, h0=None, out: Optional[Tree] = None,
                   workspace=None, stream=None) -> Tree:
        """dt_build_tree on torch's current stream (asynchronous)."""
        batch = logits.shape[0]
        if out is None:
            out = Tree.empty(batch, self.B, logits.device)
        ws = self.workspace(batch) if workspace is None else workspace
        st = self._lib.dt_build_tree(self.handle, logits.data_ptr(), batch,
                                     None if h0 is None else h0.data_ptr(), T, ws.data_ptr(),
                                     ws.numel(), ctypes.byref(out.as_c()), _stream(stream))
        if st != 0:
            _check(st)
        return out

    def build_tree_noalloc(self, logits, T: float, h0=None, out: Optional[Tree] = None,
                           stream=None) -> Tree:
        """dt_build_tree_noalloc: no workspace argument (the library's per-device
        scratch array); `out` must be given by callers that cannot allocate."""
        batch = logits.shape[0]
        if out is None:
            out = Tree.empty(batch, self.B, logits.device)
        st = self._lib.dt_build_tree_noalloc(self.handle, logits.data_ptr(), batch,
                                             None if h0 is None else h0.data_ptr(), T,
                                             ctypes.byref(out.as_c()), _stream(stream))
        if st != 0:
            _check(st)
        return out

    def _head(self, w1, w2) -> dt_domino_head:
        rank, width = w1.shape
        return dt_domino_head(_ptr(w1), _ptr(w2), width - self.d_h, rank)

    def head_workspace_size(self, batch: int, w1, w2) -> int:
        n = ctypes.c_size_t()
        hd = self._head(w1, w2)
        _check(self._lib.dt_head_workspace_size(self.handle, batch, ctypes.byref(hd), ctypes.byref(n)))
        return n.value

    def build_tree_head(self, logits, H, w1, w2, T: float, h0=None, out: Optional[Tree] = None,
                        workspace=None, stream=None) -> Tree:
        """dt_build_tree_head (Domino's own head: w1 [rank, d_H + d_h], w2 [V, rank],
        H [b, L, d_H], all in the weights dtype) on torch's current stream."""
        import torch
        batch = logits.shape[0]
        if out is None:
            out = Tree.empty(batch, self.B, logits.device)
        hd = self._head(w1, w2)
        if workspace is None:
            key = ("head", batch, hd.rank)
            if key not in self._ws:
                self._ws[key] = torch.empty(self.head_workspace_size(batch, w1, w2),
                                            dtype=torch.uint8, device=logits.device)
            workspace = self._ws[key]
        st = self._lib.dt_build_tree_head(self.handle, logits.data_ptr(), batch, H.data_ptr(),
                                          ctypes.byref(hd), None if h0 is None else h0.data_ptr(),
                                          T, workspace.data_ptr(), workspace.numel(),
                                          ctypes.byref(out.as_c()), _stream(stream))
        if st != 0:
            _check(st)
        return out

    def set_profiling(self, every: int) -> None:
        """Record stage events on every `every`-th call (0 or False: off)."""
        _check(self._lib.dt_plan_set_profiling(self.handle, int(every)))

    def stage_ms(self) -> dict:
        """Mean kernel durations (ms) over the calls profiled since set_profiling(True)."""
        ms = (ctypes.c_float * 2)()
        _check(self._lib.dt_plan_stage_ms(self.handle, ms))
        return dict(zip(STAGES, list(ms)))

    def set_adaptive_budget(self, c_draft: float = 0.0, c_verify=None) -> None:
        """CaDDTree's stopping rule with cost model (C_d, C_v(0..B)); None: fixed budget."""
        if c_verify is None:
            _check(self._lib.dt_plan_set_adaptive_budget(self.handle, 0.0, None, 0))
            return
        cv = (ctypes.c_float * len(c_verify))(*[float(x) for x in c_verify])
        _check(self._lib.dt_plan_set_adaptive_budget(self.handle, float(c_draft), cv, len(c_verify)))

    def expand_stats(self, n: int):
        """(steps, expanded) per tree of the last profiled call, as int lists."""
        steps = (ctypes.c_int32 * n)()
        expanded = (ctypes.c_int32 * n)()
        _check(self._lib.dt_plan_expand_stats(self.handle, steps, expanded, n))
        return list(steps), list(expanded)

    def close(self) -> None:
        if getattr(self, "handle", None):
            self._lib.dt_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def build_tree(marginal_logits, emb, gru_weights, correction_head, L: int, M: int, B: int,
               T: float, h0=None, max_children: int = 0, norm_mode: int = DT_NORM_TAIL,
               pos_offset: int = 0, scorer: int = DT_SCORER_COND, frontier_width: int = 0) -> Tree:
    """One-shot form of the paper's build_tree(...) -> tree (creates and drops a plan).

    gru_weights = (w_ih, w_hh, b_ih, b_hh); correction_head = (w_c, b_c).
    """
    w_ih, w_hh, b_ih, b_hh = gru_weights
    w_c, b_c = correction_head
    plan = Plan(emb, w_ih, w_hh, b_ih, b_hh, w_c, b_c, L=L, M=M, B=B,
                logits_dtype=_dtype_code(marginal_logits), max_batch=marginal_logits.shape[0],
                max_children=max_children, norm_mode=norm_mode, pos_offset=pos_offset,
                scorer=scorer, frontier_width=frontier_width)
    try:
        return plan.build_tree(marginal_logits, T, h0)
    finally:
        import torch
        torch.cuda.current_stream().synchronize()
        plan.close()


def scan_topm(logits, M: int, T: float, stream=None):
    """dt_scan_topm over a [rows, V] tensor: (ids, vals, tail_lse, row_flags)."""
    import torch
    lib = load()
    rows, V = logits.shape
    n = ctypes.c_size_t()
    _check(lib.dt_scan_workspace_size(rows, V, M, ctypes.byref(n)))
    ws = torch.empty(n.value, dtype=torch.uint8, device=logits.device)
    ids = torch.empty(rows, M, dtype=torch.int32, device=logits.device)
    vals = torch.empty(rows, M, dtype=torch.float32, device=logits.device)
    tail = torch.empty(rows, dtype=torch.float32, device=logits.device)
    flags = torch.empty(rows, dtype=torch.int32, device=logits.device)
    _check(lib.dt_scan_topm(_ptr(logits), rows, V, _dtype_code(logits), M, ctypes.c_float(T),
                            _ptr(ids), _ptr(vals), _ptr(tail), _ptr(flags), _ptr(ws), n.value,
                            _stream(stream)))
    return ids, vals, tail, flags

"""Seeded synthetic workloads for the DominoTree draft-tree builder.

This module only draws random inputs.  It holds none of the builder's
arithmetic, so both the HIP path and the CPU oracle may consume what it
produces; each side receives identical bytes.

Workloads (names follow the drafter each one is shaped like):

* ``tiny``      -- L=4, V=1024, M=8, B=8, T=0, fp32 everything, GRU d_in=d_h=64
                   with biases, head d_h->64.
* ``qwen3_4b``  -- L=16, V=151936, M=64, B=16, T=0, bf16, d_e=2560, d_h=512.
* ``qwen3_8b``  -- as above with d_e=4096 and T=1.0.
* ``budget64``  -- Qwen3-8B shapes, B=64, T=0, flattened spikes (wide trees).
* ``concurrent``-- 32 independent trees of the Qwen3-8B shape, T=0.7, per-tree
                   h0 ~ N(0, 0.1^2).
* ``deep``      -- Qwen3-8B shapes, batch 1, T=1.0, with 2-4 strong spikes
                   (+U(13,17)) per row: the top candidates dominate each row's
                   mass, so the B=16 tree grows long paths (depth 9 here) and
                   the expansion runs a long chain of dependent steps.
* ``deep_concurrent`` -- 32 trees of that kind, T=0.7, per-tree h0.

``twin_tokens(wl)`` turns a workload into one with exact structural ties:
the top token of every row gets a twin (a low-logit token given the same
embedding row and the same logit in every row), so twin paths score
identically on any builder and only the tie rules order them.

The vocabulary (151936) is Qwen3's; the block length 16 matches the b16
drafters (paper, section 4.1).  Marginal logits are 2*N(0,1) with a few
planted spikes per position, standing in for a drafter's per-position
marginals on real prompts (the paper's datasets are not used).

Generation is deterministic: every tensor is drawn from NumPy's PCG64 seeded
with ``SeedSequence([seed, tag, block])``; large tables are drawn in fixed
row blocks so a thread pool can fill them without changing the bytes.
bf16 tensors are produced as ``uint16`` bit patterns, rounded from fp32 to
nearest-even.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

import numpy as np

QWEN3_VOCAB = 151936

# tensor tags for SeedSequence
TAG_LOGITS, TAG_EMB, TAG_WIH, TAG_WHH, TAG_BIH, TAG_BHH, TAG_WC, TAG_BC, TAG_H0, TAG_SPIKE = range(10)
TAG_W1, TAG_W2, TAG_HID = 10, 11, 12

DT_F32 = 0
DT_BF16 = 1


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round-to-nearest-even) and return the uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    out = r.astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = np.uint16(0x7FC0)
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to fp32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _rng(*key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(k) for k in key]))


def _as_dtype(a32: np.ndarray, dtype: int) -> np.ndarray:
    return f32_to_bf16_bits(a32) if dtype == DT_BF16 else np.ascontiguousarray(a32, np.float32)


def _table(seed: int, tag: int, rows: int, cols: int, kind: str, scale: float, dtype: int,
           rows_per_block: int = 2048, threads: int = 8) -> np.ndarray:
    """Draw a [rows, cols] table in fixed row blocks (thread count does not change the bytes)."""
    out = np.empty((rows, cols), dtype=np.uint16 if dtype == DT_BF16 else np.float32)
    nblk = (rows + rows_per_block - 1) // rows_per_block

    def fill(i: int) -> None:
        r0 = i * rows_per_block
        r1 = min(rows, r0 + rows_per_block)
        g = _rng(seed, tag, i)
        n = (r1 - r0) * cols
        if kind == "normal":
            a = g.standard_normal(n, dtype=np.float32)
            a *= np.float32(scale)
        else:  # symmetric uniform on (-scale, scale)
            a = g.random(n, dtype=np.float32)
            a = (a * np.float32(2.0) - np.float32(1.0)) * np.float32(scale)
        out[r0:r1] = _as_dtype(a, dtype).reshape(r1 - r0, cols)

    if nblk == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(min(threads, nblk)) as ex:
            list(ex.map(fill, range(nblk)))
    return out


def peaked_logits(seed: int, tree: int, L: int, V: int, dtype: int, n_lo: int, n_hi: int,
                  spike_lo: float, spike_hi: float, fixed_spike: Optional[float] = None) -> np.ndarray:
    """[L, V] marginal logits: 2*N(0,1) plus spikes on n ~ U{n_lo..n_hi} distinct tokens per row."""
    g = _rng(seed, TAG_LOGITS, tree)
    x = g.standard_normal((L, V), dtype=np.float32) * np.float32(2.0)
    gs = _rng(seed, TAG_SPIKE, tree)
    for r in range(L):
        n = int(gs.integers(n_lo, n_hi + 1))
        toks = gs.choice(V, size=n, replace=False)
        if fixed_spike is not None:
            x[r, toks] += np.float32(fixed_spike)
        else:
            x[r, toks] += gs.uniform(spike_lo, spike_hi, size=n).astype(np.float32)
    return _as_dtype(x, dtype)


@dataclasses.dataclass
class Weights:
    """Model-side tensors (device-independent host arrays)."""
    emb: np.ndarray          # [V, d_e]
    w_ih: np.ndarray         # [3*d_h, d_e]  (PyTorch GRUCell layout, gates r,z,n)
    w_hh: np.ndarray         # [3*d_h, d_h]
    b_ih: Optional[np.ndarray]   # [3*d_h] or None
    b_hh: Optional[np.ndarray]   # [3*d_h] or None
    w_c: np.ndarray          # [d_e, d_h]    (Linear(d_h -> d_e).weight)
    b_c: Optional[np.ndarray]    # [d_e] or None
    dtype: int               # DT_F32 or DT_BF16 for every tensor above
    V: int
    d_e: int
    d_h: int


@dataclasses.dataclass
class Workload:
    name: str
    logits: np.ndarray       # [b, L, V]
    logits_dtype: int
    h0: Optional[np.ndarray] # [b, d_h] fp32 or None (zeros)
    weights: Weights
    L: int
    M: int
    B: int
    T: float
    batch: int


def make_weights(seed: int, V: int, d_e: int, d_h: int, dtype: int, gru_bias: bool,
                 head_bias: bool, emb_std: float, w_scale: float, threads: int = 8) -> Weights:
    emb = _table(seed, TAG_EMB, V, d_e, "normal", emb_std, dtype, threads=threads)
    w_ih = _table(seed, TAG_WIH, 3 * d_h, d_e, "uniform", w_scale, dtype, threads=threads)
    w_hh = _table(seed, TAG_WHH, 3 * d_h, d_h, "uniform", w_scale, dtype, threads=threads)
    w_c = _table(seed, TAG_WC, d_e, d_h, "uniform", w_scale, dtype, threads=threads)
    b_ih = _table(seed, TAG_BIH, 1, 3 * d_h, "uniform", w_scale, dtype)[0] if gru_bias else None
    b_hh = _table(seed, TAG_BHH, 1, 3 * d_h, "uniform", w_scale, dtype)[0] if gru_bias else None
    b_c = _table(seed, TAG_BC, 1, d_e, "uniform", w_scale, dtype)[0] if head_bias else None
    return Weights(emb, w_ih, w_hh, b_ih, b_hh, w_c, b_c, dtype, V, d_e, d_h)


_WEIGHT_CACHE: dict = {}


def qwen_weights(d_e: int, seed: int, threads: int = 8) -> Weights:
    key = (d_e, seed)
    if key not in _WEIGHT_CACHE:
        _WEIGHT_CACHE[key] = make_weights(seed, QWEN3_VOCAB, d_e, 512, DT_BF16, gru_bias=False,
                                          head_bias=True, emb_std=0.02,
                                          w_scale=1.0 / np.sqrt(512.0), threads=threads)
    return _WEIGHT_CACHE[key]


def tiny(seed: int = 0) -> Workload:
    L, V, M, B = 4, 1024, 8, 8
    w = make_weights(seed, V, 64, 64, DT_F32, gru_bias=True, head_bias=True, emb_std=0.02,
                     w_scale=1.0 / 8.0)
    x = peaked_logits(seed, 0, L, V, DT_F32, 3, 3, 0.0, 0.0, fixed_spike=10.0)[None]
    return Workload("tiny", x, DT_F32, None, w, L, M, B, 0.0, 1)


def qwen3_4b() -> Workload:
    w = qwen_weights(2560, 1)
    x = peaked_logits(1, 0, 16, QWEN3_VOCAB, DT_BF16, 1, 4, 6.0, 12.0)[None]
    return Workload("qwen3_4b", x, DT_BF16, None, w, 16, 64, 16, 0.0, 1)


def qwen3_8b() -> Workload:
    w = qwen_weights(4096, 2)
    x = peaked_logits(2, 0, 16, QWEN3_VOCAB, DT_BF16, 1, 4, 6.0, 12.0)[None]
    return Workload("qwen3_8b", x, DT_BF16, None, w, 16, 64, 16, 1.0, 1)


def budget64() -> Workload:
    w = qwen_weights(4096, 2)
    x = peaked_logits(3, 0, 16, QWEN3_VOCAB, DT_BF16, 4, 16, 3.0, 6.0)[None]
    return Workload("budget64", x, DT_BF16, None, w, 16, 64, 64, 0.0, 1)


def concurrent(batch: int = 32) -> Workload:
    w = qwen_weights(4096, 2)
    x = np.stack([peaked_logits(4, t, 16, QWEN3_VOCAB, DT_BF16, 1, 4, 6.0, 12.0)
                  for t in range(batch)])
    h0 = np.stack([_rng(4, TAG_H0, 1000 + t).standard_normal(512, dtype=np.float32)
                   * np.float32(0.1) for t in range(batch)])
    return Workload("concurrent", x, DT_BF16, h0, w, 16, 64, 16, 0.7, batch)


def deep() -> Workload:
    w = qwen_weights(4096, 2)
    x = peaked_logits(7, 0, 16, QWEN3_VOCAB, DT_BF16, 2, 4, 13.0, 17.0)[None]
    return Workload("deep", x, DT_BF16, None, w, 16, 64, 16, 1.0, 1)


def deep_concurrent(batch: int = 32) -> Workload:
    w = qwen_weights(4096, 2)
    x = np.stack([peaked_logits(8, t, 16, QWEN3_VOCAB, DT_BF16, 2, 4, 13.0, 17.0)
                  for t in range(batch)])
    h0 = np.stack([_rng(8, TAG_H0, 1000 + t).standard_normal(512, dtype=np.float32)
                   * np.float32(0.1) for t in range(batch)])
    return Workload("deep_concurrent", x, DT_BF16, h0, w, 16, 64, 16, 0.7, batch)


WORKLOADS = {
    "tiny": tiny,
    "qwen3_4b": qwen3_4b,
    "qwen3_8b": qwen3_8b,
    "budget64": budget64,
    "concurrent": concurrent,
    "deep": deep,
    "deep_concurrent": deep_concurrent,
}


def twin_tokens(wl: Workload) -> Workload:
    """A copy of `wl` whose rows' top tokens have twins.

    For every distinct token a that tops some row of some tree, a twin b is
    taken from the tokens that top no row and sit lowest in row 0 of tree 0;
    E[b] is set to E[a] and, in every row of every tree, the logit of b to
    that of a.  The embedding table is copied (the cached one is untouched).
    """
    x = wl.logits.copy()
    flat = x.reshape(-1, x.shape[-1])
    vals = bf16_bits_to_f32(flat) if wl.logits_dtype == DT_BF16 else flat
    tops = sorted({int(np.argmax(r)) for r in vals})
    row0 = vals[0]
    spare = [int(v) for v in np.argsort(row0, kind="stable") if int(v) not in set(tops)]
    w = wl.weights
    emb = w.emb.copy()
    for a, b in zip(tops, spare):
        emb[b] = emb[a]
        flat[:, b] = flat[:, a]
    wt = dataclasses.replace(w, emb=emb)
    return Workload(wl.name + "_twins", x, wl.logits_dtype, wl.h0, wt, wl.L, wl.M, wl.B, wl.T,
                    wl.batch)


@dataclasses.dataclass
class DominoHead:
    """Domino's own correction head (section 2.3): rank-r bottleneck with SiLU."""
    w1: np.ndarray   # [rank, d_H + d_h]  Linear(d_H + d_h -> rank).weight; columns [0, d_H) take H
    w2: np.ndarray   # [V, rank]          Linear(rank -> V).weight
    dtype: int
    d_H: int
    rank: int


def domino_head(seed: int, V: int, d_H: int, d_h: int, rank: int, dtype: int,
                w1_scale: Optional[float] = None, w2_scale: Optional[float] = None,
                threads: int = 8) -> DominoHead:
    """Uniform weights at PyTorch Linear's fan-in scale unless scales are given."""
    s1 = 1.0 / np.sqrt(d_H + d_h) if w1_scale is None else w1_scale
    s2 = 1.0 / np.sqrt(rank) if w2_scale is None else w2_scale
    w1 = _table(seed, TAG_W1, rank, d_H + d_h, "uniform", s1, dtype, threads=threads)
    w2 = _table(seed, TAG_W2, V, rank, "uniform", s2, dtype, threads=threads)
    return DominoHead(w1, w2, dtype, d_H, rank)


def hidden_states(seed: int, batch: int, L: int, d_H: int, dtype: int, std: float = 1.0) -> np.ndarray:
    """[batch, L, d_H] drafter hidden states H_d, standard normal times std."""
    h = _rng(seed, TAG_HID, 0).standard_normal((batch, L, d_H), dtype=np.float32) * np.float32(std)
    return _as_dtype(h, dtype)


def random_small(seed: int, *, batch: int, L: int, V: int, M: int, B: int, T: float,
                 d_e: int, d_h: int, dtype: int = DT_F32, logits_dtype: Optional[int] = None,
                 gru_bias: bool = True, head_bias: bool = True, h0: bool = False,
                 emb_std: float = 0.5, w_scale: float = 0.5, logit_scale: float = 2.0,
                 spikes: int = 2, spike: float = 4.0) -> Workload:
    """Small random workload for parity sweeps (large corrections so paths really differ)."""
    w = make_weights(seed, V, d_e, d_h, dtype, gru_bias, head_bias, emb_std, w_scale)
    ldt = dtype if logits_dtype is None else logits_dtype
    g = _rng(seed, TAG_LOGITS, 99)
    x = g.standard_normal((batch, L, V), dtype=np.float32) * np.float32(logit_scale)
    for t in range(batch):
        for r in range(L):
            toks = g.choice(V, size=min(spikes, V), replace=False)
            x[t, r, toks] += np.float32(spike) * g.random(len(toks), dtype=np.float32)
    hh = None
    if h0:
        hh = _rng(seed, TAG_H0, 0).standard_normal((batch, d_h), dtype=np.float32) * np.float32(0.5)
    return Workload(f"random{seed}", _as_dtype(x, ldt), ldt, hh, w, L, M, B, T, batch)


# generator settings of each workload's logits, for drawing more buffers of the same kind
LOGIT_RECIPES = {
    "tiny": dict(seed=0, dtype=DT_F32, L=4, V=1024, n_lo=3, n_hi=3, lo=0.0, hi=0.0, fixed=10.0),
    "qwen3_4b": dict(seed=1, dtype=DT_BF16, L=16, V=QWEN3_VOCAB, n_lo=1, n_hi=4, lo=6.0, hi=12.0,
                     fixed=None),
    "qwen3_8b": dict(seed=2, dtype=DT_BF16, L=16, V=QWEN3_VOCAB, n_lo=1, n_hi=4, lo=6.0, hi=12.0,
                     fixed=None),
    "budget64": dict(seed=3, dtype=DT_BF16, L=16, V=QWEN3_VOCAB, n_lo=4, n_hi=16, lo=3.0, hi=6.0,
                     fixed=None),
    "concurrent": dict(seed=4, dtype=DT_BF16, L=16, V=QWEN3_VOCAB, n_lo=1, n_hi=4, lo=6.0,
                       hi=12.0, fixed=None),
    "deep": dict(seed=7, dtype=DT_BF16, L=16, V=QWEN3_VOCAB, n_lo=2, n_hi=4, lo=13.0, hi=17.0,
                 fixed=None),
    "deep_concurrent": dict(seed=8, dtype=DT_BF16, L=16, V=QWEN3_VOCAB, n_lo=2, n_hi=4, lo=13.0,
                            hi=17.0, fixed=None),
}


def logits_buffer(name: str, index: int, batch: int, threads: int = 8) -> np.ndarray:
    """[batch, L, V] logits for buffer `index` of a workload (buffer 0 = the workload's own).

    Tree t of buffer i is drawn with tree index i*batch + t, so buffers never repeat.
    """
    r = LOGIT_RECIPES[name]

    def one(t: int) -> np.ndarray:
        return peaked_logits(r["seed"], index * batch + t, r["L"], r["V"], r["dtype"], r["n_lo"],
                             r["n_hi"], r["lo"], r["hi"], fixed_spike=r["fixed"])

    with ThreadPoolExecutor(min(threads, batch)) as ex:
        return np.stack(list(ex.map(one, range(batch))))

"""Unit pins of the oracle's building blocks against library routines and brute force."""
import math

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from paper_2607_08642_amd import synth


@pytest.mark.parametrize("bias", [True, False])
def test_gru_cell_matches_torch_grucell(bias):
    # Domino's encoder is a GRU (section 2.3); the gate convention is GRUCell's.
    rng = np.random.default_rng(1)
    d_in, d_h, k = 7, 5, 4
    w_ih = rng.standard_normal((3 * d_h, d_in))
    w_hh = rng.standard_normal((3 * d_h, d_h))
    b_ih = rng.standard_normal(3 * d_h) if bias else None
    b_hh = rng.standard_normal(3 * d_h) if bias else None
    h = rng.standard_normal(d_h)
    xs = rng.standard_normal((k, d_in))
    got = oracle.gru_cell(h, xs, w_ih, w_hh, b_ih, b_hh)
    cell = torch.nn.GRUCell(d_in, d_h, bias=bias).double()
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(w_ih))
        cell.weight_hh.copy_(torch.from_numpy(w_hh))
        if bias:
            cell.bias_ih.copy_(torch.from_numpy(b_ih))
            cell.bias_hh.copy_(torch.from_numpy(b_hh))
        want = cell(torch.from_numpy(xs), torch.from_numpy(h)[None].expand(k, d_h)).numpy()
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-13)


def _brute_topm(x, M):
    return sorted(range(len(x)), key=lambda v: (-x[v], v))[:M]


@pytest.mark.parametrize("seed", range(6))
def test_scan_row_matches_brute_force_with_ties(seed):
    # Alg. 1 step 1: top-M by (logit desc, id asc); ties are frequent after bf16 rounding.
    rng = np.random.default_rng(seed)
    V, M = 97, 11
    x = np.round(rng.standard_normal(V) * 2, 1)      # coarse grid -> many exact ties
    x[rng.choice(V, 5, replace=False)] = -np.inf
    tau = [1.0, 0.7, 2.5][seed % 3]
    ids, xs, R = oracle.scan_row(x, M, tau)
    want = _brute_topm(x.tolist(), M)
    assert ids.tolist() == want
    assert xs.tolist() == [x[v] for v in want]
    assert ids.tolist() == np.lexsort((np.arange(V), -x))[:M].tolist()
    rest = [v for v in range(V) if v not in set(want)]
    assert R == pytest.approx(scipy.special.logsumexp(x[rest] / tau), rel=1e-13)


def test_scan_row_full_vocab_has_empty_tail():
    x = np.array([0.5, -1.0, 3.0, -np.inf])
    ids, xs, R = oracle.scan_row(x, 4, 1.0)
    assert ids.tolist() == [2, 0, 1, 3]
    assert R == -math.inf


def test_scan_row_all_equal_takes_lowest_ids():
    x = np.zeros(50)
    ids, _, R = oracle.scan_row(x, 7, 1.0)
    assert ids.tolist() == list(range(7))
    assert R == pytest.approx(math.log(43))


def test_logsumexp_matches_scipy():
    rng = np.random.default_rng(3)
    a = rng.standard_normal(1000) * 30
    assert oracle.logsumexp(a) == pytest.approx(scipy.special.logsumexp(a), rel=1e-14)
    assert oracle.logsumexp(np.array([])) == -math.inf
    assert oracle.logsumexp(np.array([-np.inf, -np.inf])) == -math.inf


def test_bf16_widening_matches_torch():
    rng = np.random.default_rng(4)
    a = (rng.standard_normal(10000) * 5).astype(np.float32)
    bits = synth.f32_to_bf16_bits(a)
    want = torch.from_numpy(a).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(oracle.widen(bits, oracle.DT_BF16), want)


def test_effective_temperature():
    assert oracle.effective_temperature(0.0) == 1.0
    assert oracle.effective_temperature(0.7) == 0.7

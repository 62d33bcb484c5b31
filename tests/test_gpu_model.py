"""One model, several plans (dt_model_create, dt_plan_create_from_model), through
the C ABI.

Plans of different shapes and options over one model's tables must build the
same trees, bit for bit, as plans that fold the vocabulary themselves
(dt_plan_create), and those trees match the oracle; the tables stay alive while
a plan uses them after the model handle is released, and a plan made from a
model allocates none of the vocabulary tables again.
"""
import numpy as np
import pytest
import torch

from gpu_util import compare_tree, to_dev
from paper_2607_08642_amd import binding, synth

pytestmark = pytest.mark.gpu
FIELDS = ("tokens", "parents", "depth", "position_ids", "mask", "scores", "n_nodes", "status")


def weights_on_device(wl):
    w = wl.weights
    return [to_dev(a, w.dtype) for a in (w.emb, w.w_ih, w.w_hh, w.b_ih, w.b_hh, w.w_c, w.b_c)]


def run(plan, logits, T, h0):
    tree = plan.build_tree(logits, T, h0)
    torch.cuda.synchronize()
    return {k: getattr(tree, k).cpu().numpy() for k in FIELDS}


def test_plans_of_several_shapes_share_one_model():
    wl = synth.random_small(61, batch=3, L=6, V=3000, M=32, B=24, T=0.7, d_e=64, d_h=64,
                            dtype=synth.DT_BF16, h0=True)
    tensors = weights_on_device(wl)
    model = binding.Model(*tensors)
    h0 = torch.from_numpy(wl.h0.astype(np.float32)).cuda()
    shapes = [dict(L=6, M=32, B=24), dict(L=4, M=16, B=8, max_children=3),
              dict(L=6, M=32, B=24, scorer=binding.DT_SCORER_MARG), dict(L=5, M=8, B=40, pos_offset=3)]
    try:
        for kw in shapes:
            print(f"[model] shape {kw}", flush=True)
            L = kw["L"]
            logits = to_dev(np.ascontiguousarray(wl.logits[:, :L]), wl.logits_dtype)
            shared = binding.Plan.from_model(model, logits_dtype=wl.logits_dtype, max_batch=3, **kw)
            own = binding.Plan(*tensors, logits_dtype=wl.logits_dtype, max_batch=3, **kw)
            try:
                a = run(shared, logits, wl.T, h0)
                b = run(own, logits, wl.T, h0)
            finally:
                shared.close()
                own.close()
            for k in FIELDS:
                np.testing.assert_array_equal(a[k], b[k], err_msg=f"{kw} {k}")
            if kw.get("scorer", 0) == 0 and L == wl.L and kw["M"] == wl.M and kw["B"] == wl.B:
                okw = dict(max_children=0, norm_mode=0, pos_offset=0, scorer=0)
                for t in range(wl.batch):
                    compare_tree(wl, t, a, okw, name="model-shared")
    finally:
        model.close()


def test_tables_outlive_the_model_handle():
    wl = synth.random_small(62, batch=2, L=5, V=2000, M=16, B=12, T=1.0, d_e=64, d_h=64)
    tensors = weights_on_device(wl)
    model = binding.Model(*tensors)
    p1 = binding.Plan.from_model(model, L=wl.L, M=wl.M, B=wl.B, logits_dtype=wl.logits_dtype,
                                 max_batch=2)
    p2 = binding.Plan.from_model(model, L=wl.L, M=wl.M, B=wl.B, logits_dtype=wl.logits_dtype,
                                 max_batch=2)
    model.close()            # the plans keep the tables
    del tensors              # (the weights are not read after the model is built)
    torch.cuda.empty_cache()
    logits = to_dev(wl.logits, wl.logits_dtype)
    try:
        a = run(p1, logits, wl.T, None)
        p1.close()
        b = run(p2, logits, wl.T, None)
    finally:
        p1.close()
        p2.close()
    for k in FIELDS:
        np.testing.assert_array_equal(a[k], b[k], err_msg=k)
    okw = dict(max_children=0, norm_mode=0, pos_offset=0, scorer=0)
    for t in range(wl.batch):
        compare_tree(wl, t, a, okw, name="model-released")


def test_plans_from_a_model_fold_nothing_again():
    # V = 50000, d_h = 64: the tables take V * (4 d_h + 1) * 4 = 51.4 MB
    wl = synth.random_small(63, batch=1, L=4, V=50000, M=16, B=8, T=0.0, d_e=64, d_h=64)
    tensors = weights_on_device(wl)
    table = 50000 * (4 * 64 + 1) * 4
    torch.cuda.synchronize()
    free0 = torch.cuda.mem_get_info()[0]
    model = binding.Model(*tensors)
    free1 = torch.cuda.mem_get_info()[0]
    plans = [binding.Plan.from_model(model, L=wl.L, M=m, B=wl.B, logits_dtype=wl.logits_dtype)
             for m in (8, 16, 32)]
    free2 = torch.cuda.mem_get_info()[0]
    print(f"[model] tables {table / 1e6:.1f} MB: model took {(free0 - free1) / 1e6:.1f} MB, "
          f"three plans {(free1 - free2) / 1e6:.1f} MB", flush=True)
    try:
        assert free0 - free1 >= 0.9 * table
        assert free1 - free2 < 0.1 * table
    finally:
        for p in plans:
            p.close()
        model.close()
    torch.cuda.synchronize()
    free3 = torch.cuda.mem_get_info()[0]
    assert free3 - free2 >= 0.9 * table     # freed with the last reference

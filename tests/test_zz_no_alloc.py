"""dt_build_tree_noalloc (the entry point for callers that cannot allocate)
against dt_build_tree with a caller workspace, through the C ABI.

Two calls in a row on the library's scratch array, the second with a smaller
batch, must reproduce dt_build_tree's trees bit for bit; a batch whose
workspace exceeds the 32 MiB array is rejected on the host.
"""
import numpy as np
import pytest
import torch

from gpu_util import to_dev
from paper_2607_08642_amd import binding, synth

pytestmark = pytest.mark.gpu

FIELDS = ("tokens", "parents", "depth", "position_ids", "mask", "scores", "n_nodes", "status")


def snap(tree):
    return {k: getattr(tree, k).cpu().numpy().copy() for k in FIELDS}


def test_noalloc_matches_workspace_path():
    wl = synth.deep_concurrent()
    w = wl.weights
    d = w.dtype
    print(f"[noalloc] deep_concurrent batch={wl.batch}", flush=True)
    emb = to_dev(w.emb, d)
    plan = binding.Plan(emb, to_dev(w.w_ih, d), to_dev(w.w_hh, d), None, None, to_dev(w.w_c, d),
                        to_dev(w.b_c, d), L=wl.L, M=wl.M, B=wl.B, logits_dtype=wl.logits_dtype,
                        max_batch=64)
    try:
        logits = to_dev(wl.logits, wl.logits_dtype)
        h0 = torch.from_numpy(wl.h0).cuda()
        for batch in (32, 5):     # the second call on the scratch array is smaller
            x, hh = logits[:batch].contiguous(), h0[:batch].contiguous()
            out = binding.Tree.empty(batch, wl.B, "cuda")
            plan.build_tree_noalloc(x, wl.T, hh, out=out)
            torch.cuda.synchronize()
            got = snap(out)
            ref = snap(plan.build_tree(x, wl.T, hh))
            torch.cuda.synchronize()
            for k in FIELDS:
                np.testing.assert_array_equal(got[k], ref[k], err_msg=f"batch {batch}: {k}")
            assert (got["n_nodes"] == wl.B).all()
            print(f"[noalloc] batch {batch}: identical to dt_build_tree", flush=True)
        # 64 trees need more than the scratch array holds: rejected before any launch
        assert plan.workspace_size(64) > 32 << 20
        big = torch.zeros(64, wl.L, w.V, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(binding.DTError) as e:
            plan.build_tree_noalloc(big, wl.T)
        assert e.value.status == -5 and b"scratch" in binding.load().dt_last_error()
    finally:
        plan.close()

"""The bounded waits of the workgroups that build one tree together
(dt_options.debug_spin_limit; DT_TREE_TIMEOUT).

With a spin limit of one poll the members of a tree give up waiting for one
another almost at once: every kernel must still exit normally, a tree whose
wait gave up must come out empty and flagged, any other tree must be the
oracle's, and a plan with the default limit must afterwards build correct
trees on the same device.  The condition is forced from the host; no kernel
faults or hangs.
"""
import numpy as np
import pytest

from gpu_util import DeviceWorkload, compare_tree
from paper_2607_08642_amd import binding, synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["deep", "deep_concurrent"])
def test_spin_limit_gives_up_cleanly(name):
    wl = synth.WORKLOADS[name]()
    print(f"[timeout] {name} batch={wl.batch} spin limit 1", flush=True)
    dw = DeviceWorkload(wl, debug_spin_limit=1)
    try:
        got = dw.run()
    finally:
        dw.close()
    timed_out = 0
    for t in range(wl.batch):
        st = int(got["status"][t])
        if st & binding.DT_TREE_TIMEOUT:
            timed_out += 1
            assert int(got["n_nodes"][t]) == 0
            assert (got["tokens"][t] == -1).all() and (got["mask"][t] == 0).all()
            assert (got["scores"][t] == -np.inf).all()
        elif t < 3:
            compare_tree(wl, t, got, {}, tol=1e-4, name=f"timeout-{name}")
    print(f"[timeout] {name}: {timed_out} of {wl.batch} trees timed out", flush=True)
    assert timed_out >= 1
    # the default limit on the same device: correct trees
    dw = DeviceWorkload(wl)
    try:
        again = dw.run()
    finally:
        dw.close()
    assert not (again["status"] & binding.DT_TREE_TIMEOUT).any()
    for t in range(min(wl.batch, 2)):
        compare_tree(wl, t, again, {}, tol=1e-4, name=f"after-timeout-{name}")

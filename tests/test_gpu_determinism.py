"""Run-twice determinism of the GPU path.

One flipped eviction changes every later step of a head, so the kernels must
decide identically on identical inputs however their blocks are scheduled:
the fp64 eviction scores and grouping mass are summed in a fixed order, the
radix selection takes equal keys in position order, and the split-K merge of
a chunked layer combines its partial results in a fixed tree over the chunk
indices (left before right) whichever chunk arrives first.  Two fresh sessions over the same inputs must give bitwise-equal
labels, n*, budgets, retained sets and attention outputs.
"""
import pytest
import torch

from paper_2605_20600_amd import workloads as W
from paper_2605_20600_amd.runner import DeviceInputs, new_session, run_generation

pytestmark = pytest.mark.gpu


def _steps(wl, n_steps):
    t_g, P = wl.group_threshold - 1, wl.period
    s = set(range(0, n_steps, 97)) | {t_g, t_g + 1, n_steps - 1}
    s |= {t for t in range(t_g, n_steps, P)} | {t + 1 for t in range(t_g, n_steps - 1, P)}
    return sorted(t for t in s if t < n_steps)


def _run(wl, inp, steps, n_steps):
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps, steps=n_steps)
    torch.cuda.synchronize()
    sess.close()
    return res


@pytest.mark.parametrize("wl,n_steps", [
    (W.LUMINA768.with_(layers=2), None),
    (W.LUMINA1024.with_(layers=1), 500 + 3 * 65 + 2),
], ids=["lumina768-2layers-whole", "lumina1024-chunked"])
def test_run_twice_bitwise(wl, n_steps):
    n_steps = wl.num_visual if n_steps is None else n_steps
    steps = _steps(wl, n_steps)
    inp = DeviceInputs(wl)
    a = _run(wl, inp, steps, n_steps)
    b = _run(wl, inp, steps, n_steps)
    for key in ("is_local", "n_star", "budgets"):
        for l in a[key]:
            assert torch.equal(a[key][l], b[key][l]), (key, l)
    for (t, l) in a["snap"]:
        for x, y in zip(a["snap"][(t, l)], b["snap"][(t, l)]):
            assert torch.equal(x, y), ("retained", t, l)
    for (t, l) in a["out"]:
        assert torch.equal(a["out"][(t, l)], b["out"][(t, l)]), ("out", t, l)
    print(f"{wl.name}: {len(steps)} steps x {len(inp.layers)} layers bitwise identical over two "
          f"runs", flush=True)


def test_deep_merge_trees_run_twice_bitwise():
    # chunk counts 1..24 per head (merge trees of up to five levels)
    import numpy as np
    from test_gpu_edges import DEEP_TREE_BUDGETS, DEEP_TREE_STEPS, DEEP_TREES
    wl = DEEP_TREES
    inp = DeviceInputs(wl, layers=[0])
    inp.override[0] = torch.as_tensor(np.asarray(DEEP_TREE_BUDGETS, dtype=np.int32).reshape(-1),
                                      device="cuda")
    a = _run(wl, inp, DEEP_TREE_STEPS, wl.num_visual)
    b = _run(wl, inp, DEEP_TREE_STEPS, wl.num_visual)
    for (t, l) in a["out"]:
        assert torch.equal(a["out"][(t, l)], b["out"][(t, l)]), ("out", t, l)
    for (t, l) in a["snap"]:
        for x, y in zip(a["snap"][(t, l)], b["snap"][(t, l)]):
            assert torch.equal(x, y), ("retained", t, l)

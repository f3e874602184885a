"""GPU <-> oracle parity through the C ABI.

Bar: labels, n*, budgets and retained position sets bit-exact; attention
outputs within max-abs 2e-2 of the fp64 oracle (bf16 storage, fp32
accumulation)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_20600_amd import synth, workloads as W
from paper_2605_20600_amd.runner import DeviceInputs, new_session, run_generation

pytestmark = pytest.mark.gpu
ATOL = 2e-2


def _say(*a):
    print(*a, flush=True)


def _check_slice(wl, res, layer, b, steps, ref=None, heads=None):
    """Compares one (layer, b) slice of a GPU run with the oracle."""
    H = wl.heads
    heads = list(range(H)) if heads is None else heads
    if ref is None:
        ref = oracle.simulate(wl, layer, b, heads=heads, snap_steps=steps)
    sl = slice(b * H, (b + 1) * H)
    assert np.array_equal(res["is_local"][layer][sl].cpu().numpy(), ref["labels"]), "labels"
    assert np.array_equal(res["n_star"][layer][sl].cpu().numpy(), ref["n_star"]), "n_star"
    assert np.array_equal(res["budgets"][layer][sl].cpu().numpy(), ref["budgets"]), "budgets"
    worst = 0.0
    for i, t in enumerate(steps):
        mask, count = res["snap"][(t, layer)]
        mask = mask[sl].cpu().numpy()
        out = res["out"][(t, layer)][b].cpu().double().numpy()
        for h in heads:
            exp_mask = ref["snaps"][h][i]
            assert np.array_equal(mask[h], exp_mask), (layer, b, h, t)
            assert int(count[b * H + h]) == int(exp_mask.sum())
            err = float(np.abs(out[h] - ref["out"][h][t]).max())
            worst = max(worst, err)
            assert err <= ATOL, (layer, b, h, t, err)
    return worst, ref


def test_generator_bitwise_cpu_gpu():
    wl = W.LUMINA768
    for layer, t0, t1 in ((0, 0, 3), (17, 2000, 2003)):
        g = synth.visual_qkv(wl, layer, t0, t1, "cuda")
        c = synth.visual_qkv(wl, layer, t0, t1, "cpu")
        for x, y in zip(g, c):
            assert torch.equal(x.cpu(), y)
    g = synth.prefix_kv(wl, 5, "cuda")
    c = synth.prefix_kv(wl, 5, "cpu")
    assert all(torch.equal(x.cpu(), y) for x, y in zip(g, c))


def test_tiny_full_generation_every_step():
    wl = W.TINY
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
    torch.cuda.synchronize()
    worst, _ = _check_slice(wl, res, 0, 0, steps)
    _say(f"tiny: every step bit-exact, max |out - oracle| = {worst:.3e}")


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_tiny_other_seeds(seed):
    wl = W.TINY
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl, seed=seed)
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
    torch.cuda.synchronize()
    ref = oracle.simulate(wl, 0, 0, snap_steps=steps, seed=seed)
    _check_slice(wl, res, 0, 0, steps, ref=ref)


def test_tiny_full_budget_is_full_attention():
    # every budget = N: compressed attention must equal full attention
    wl = W.TINY.with_(budget_mode=W.BUDGET_OVERRIDE)
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl)
    inp.override[0] = torch.full((wl.heads,), wl.num_visual, dtype=torch.int32, device="cuda")
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
    torch.cuda.synchronize()
    for h in range(wl.heads):
        q, k, v, kc, vc = synth.head_inputs(wl, 0, 0, h)
        for t in (0, 63, 64, 100, 255):
            ref = oracle.attention(q[t], torch.cat([kc, k[: t + 1]]), torch.cat([vc, v[: t + 1]]))
            got = res["out"][(t, 0)][0, h].cpu().double().numpy()
            assert np.abs(got - ref).max() <= ATOL
            assert int(res["snap"][(t, 0)][1][h]) == t + 1


def _lumina_steps(wl):
    t_g, P, N = wl.group_threshold - 1, wl.period, wl.num_visual
    return sorted({0, 1, 127, t_g - 1, t_g, t_g + 1, t_g + P - 1, t_g + P, t_g + P + 1,
                   1000, N - 2, N - 1})


@pytest.mark.parametrize("rho", [(1, 8), (1, 4)])
def test_lumina768_two_layers_sampled(rho):
    # full head count and batch, two of the 32 layers, every step of the generation
    wl = W.LUMINA768.with_(rho=rho)
    steps = _lumina_steps(wl)
    inp = DeviceInputs(wl, layers=[0, 31])
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
    torch.cuda.synchronize()
    for (layer, b) in ((0, 0), (31, 7)):
        worst, ref = _check_slice(wl, res, layer, b, steps)
        _say(f"lumina768 rho={rho} layer {layer} b {b}: bit-exact, max err {worst:.3e}, "
             f"label margin min {np.abs(ref['mass_window'] - wl.tau).min():.3e}")
    # labels, n* and budgets of every head of both layers
    for layer in (0, 31):
        g = oracle.group_layer(wl, layer)
        assert np.array_equal(res["is_local"][layer].cpu().numpy(), g["labels"].reshape(-1))
        assert np.array_equal(res["n_star"][layer].cpu().numpy(), g["n_star"].reshape(-1))
        assert np.array_equal(res["budgets"][layer].cpu().numpy(), g["budgets"].reshape(-1))

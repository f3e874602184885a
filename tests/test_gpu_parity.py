"""GPU <-> oracle parity through the C ABI.

Bar: labels, n*, budgets and retained position sets bit-exact; attention
outputs within max-abs 2e-2 of the fp64 oracle (bf16 storage, fp32
accumulation).  Full-shape workloads are checked on sampled (layer, batch row)
slices, every head of a slice, at sampled steps that include the grouping step
and update steps; labels, n* and budgets on every head of the layers run."""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_20600_amd import binding as B, synth, workloads as W
from paper_2605_20600_amd.runner import (DeviceInputs, new_session, run_generation,
                                         run_generation_native)
from parity_report import assert_same_retained

pytestmark = pytest.mark.gpu
ATOL = 2e-2


def _say(*a):
    print(*a, flush=True)


def _check_slice(wl, res, layer, b, steps, ref=None):
    """Compares one (layer, b) slice of a GPU run with the oracle."""
    H = wl.heads
    if ref is None:
        ref = oracle.simulate(wl, layer, b, snap_steps=steps)
    sl = slice(b * H, (b + 1) * H)
    assert np.array_equal(res["is_local"][layer][sl].cpu().numpy(), ref["labels"]), "labels"
    assert np.array_equal(res["n_star"][layer][sl].cpu().numpy(), ref["n_star"]), "n_star"
    assert np.array_equal(res["budgets"][layer][sl].cpu().numpy(), ref["budgets"]), "budgets"
    masks = [res["snap"][(t, layer)][0][sl].cpu().numpy() for t in steps]
    assert_same_retained(steps, masks, ref, range(H), wl.period, wl.group_threshold - 1,
                         f"{wl.name} layer {layer} b {b}:")
    worst = 0.0
    for i, t in enumerate(steps):
        count = res["snap"][(t, layer)][1][sl].cpu().numpy()
        out = res["out"][(t, layer)][b].cpu().double().numpy()
        for h in range(H):
            exp_mask = ref["snaps"][h][i]
            assert int(count[h]) == int(exp_mask.sum())
            err = float(np.abs(out[h] - ref["out"][h][t]).max())
            worst = max(worst, err)
            assert err <= ATOL, (layer, b, h, t, err)
    return worst, ref


def _steps(wl, extra=()):
    t_g, P, N = wl.group_threshold - 1, wl.period, wl.num_visual
    s = {0, 1, t_g - 1, t_g, t_g + 1, t_g + P - 1, t_g + P, t_g + P + 1, N // 2, N - 2, N - 1}
    return sorted(x for x in s.union(extra) if 0 <= x < N)


def _run_and_check(wl, layers, slices, steps, fused=True, all_heads=True, strategy=0,
                   n_steps=None):
    inp = DeviceInputs(wl, layers=layers)
    sess = new_session(wl, attn_strategy=strategy)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps, fused=fused,
                         record_layers=sorted({l for l, _ in slices}), steps=n_steps)
    torch.cuda.synchronize()
    for (layer, b) in slices:
        worst, ref = _check_slice(wl, res, layer, b, steps)
        gaps = [st["min_gap"] for st in ref["stats"].values()]
        _say(f"{wl.name} rho={wl.rho} fused={fused} strategy={strategy} layer {layer} b {b}: bit-exact; "
             f"max err {worst:.2e}; min label margin "
             f"{np.abs(ref['mass_window'] - wl.tau).min():.2e}; min eviction score gap "
             f"{min(gaps):.2e}")
    if all_heads:
        for layer in layers:
            g = oracle.group_layer(wl, layer)
            assert np.array_equal(res["is_local"][layer].cpu().numpy(), g["labels"].reshape(-1))
            assert np.array_equal(res["n_star"][layer].cpu().numpy(), g["n_star"].reshape(-1))
            assert np.array_equal(res["budgets"][layer].cpu().numpy(), g["budgets"].reshape(-1))
    return res


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


@pytest.mark.parametrize("fused", [True, False])
def test_tiny_full_generation_every_step(fused):
    wl = W.TINY
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps, fused=fused)
    torch.cuda.synchronize()
    worst, _ = _check_slice(wl, res, 0, 0, steps)
    _say(f"tiny fused={fused}: every step bit-exact, max |out - oracle| = {worst:.3e}")


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


def test_tiny_linear_uniform_budgets():
    # every head labelled global: the uniform-budget layout of the line-based
    # baseline the paper compares against, through the same calls
    wl = W.TINY
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    lab = {0: torch.zeros(wl.heads, dtype=torch.uint8, device="cuda")}
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps, label_override=lab)
    torch.cuda.synchronize()
    ref = oracle.simulate(wl, 0, 0, snap_steps=steps, label_override=[0] * wl.heads)
    assert list(ref["budgets"]) == [wl.num_visual * wl.rho[0] // wl.rho[1]] * wl.heads
    _check_slice(wl, res, 0, 0, steps, ref=ref)


@pytest.mark.parametrize("rho", [(1, 8), (1, 6), (1, 4)])
def test_lumina768_sampled(rho):
    wl = W.LUMINA768.with_(rho=rho)
    # steps 127 and 200: the full cache in half and three-quarter passes
    _run_and_check(wl, [0, 31], [(0, 0), (31, 7)], _steps(wl, extra=(127, 200, 1000)))


@pytest.mark.parametrize("seed", [7, 2024])
def test_lumina768_other_data_seeds(seed):
    # the full Lumina-768 shape on other synthetic draws: one layer, two batch
    # rows, every head, at the sampled steps (grouping, updates, the end)
    wl = W.LUMINA768
    layer = 11
    steps = _steps(wl, extra=(800, 1600))
    inp = DeviceInputs(wl, layers=[layer], seed=seed)
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
    torch.cuda.synchronize()
    for b in (2, 6):
        ref = oracle.simulate(wl, layer, b, snap_steps=steps, seed=seed)
        worst, _ = _check_slice(wl, res, layer, b, steps, ref=ref)
        _say(f"lumina768 seed {seed} layer {layer} b {b}: bit-exact; max err {worst:.2e}")


def test_lumina768_separate_calls():
    wl = W.LUMINA768
    _run_and_check(wl, [5], [(5, 3)], _steps(wl), fused=False, all_heads=False)


def test_lumina1024_separate_calls():
    # fewer heads than CUs: the chunked attention without a fused append
    wl = W.LUMINA1024
    _run_and_check(wl, [7], [(7, 2)], _steps(wl), fused=False, all_heads=False)


def test_janus7b_total_budget_sampled():
    wl = W.JANUS7B
    _run_and_check(wl, [0, 29], [(0, 0), (29, 15)], _steps(wl, extra=(200, 400)))


def test_lumina1024_override_split_heads():
    # 4 x 32 = 128 heads per layer < 256 compute units: each head is cut into
    # chunks of one pass by the layer's chunk table and merged
    wl = W.LUMINA1024
    _run_and_check(wl, [0, 31], [(0, 0), (31, 3)], _steps(wl, extra=(2000, 3000)))


def test_stress_update_every_step():
    wl = W.STRESS
    _run_and_check(wl, [0], [(0, 0), (0, 63)], _steps(wl, extra=(310, 1500)))


@pytest.mark.parametrize("wl", [W.TINY, W.LUMINA768.with_(layers=2)], ids=["tiny", "lumina2"])
def test_native_step_loop(wl):
    # the library's own step loop gives the same final state as the oracle
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    outs = {l: torch.empty((wl.batch, wl.heads, wl.head_dim), dtype=torch.float32, device="cuda")
            for l in range(wl.layers)}
    res = run_generation_native(sess, inp, outs)
    N = wl.num_visual
    for l in range(wl.layers):
        mask, count = sess.export_retained(l)
        torch.cuda.synchronize()
        ref = oracle.simulate(wl, l, 0, snap_steps=[N - 1])
        H = wl.heads
        assert np.array_equal(res["is_local"][l][:H].cpu().numpy(), ref["labels"])
        assert np.array_equal(res["budgets"][l][:H].cpu().numpy(), ref["budgets"])
        out = outs[l][0].cpu().double().numpy()
        for h in range(H):
            assert np.array_equal(mask[h].cpu().numpy(), ref["snaps"][h][0]), (l, h)
            assert np.abs(out[h] - ref["out"][h][N - 1]).max() <= ATOL


STRATEGIES = [B.HEADKV_ATTN_PADDED, B.HEADKV_ATTN_GROUPED]
STRATEGY_IDS = ["padded", "grouped"]


@pytest.mark.parametrize("strategy", STRATEGIES, ids=STRATEGY_IDS)
@pytest.mark.parametrize("fused", [True, False])
def test_tiny_strategies_every_step(strategy, fused):
    # the paper's other two attention strategies give the oracle's outputs
    wl = W.TINY
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl)
    sess = new_session(wl, attn_strategy=strategy)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps, fused=fused)
    torch.cuda.synchronize()
    worst, _ = _check_slice(wl, res, 0, 0, steps)
    _say(f"tiny strategy={strategy} fused={fused}: every step bit-exact, max err {worst:.3e}")


@pytest.mark.parametrize("strategy", STRATEGIES, ids=STRATEGY_IDS)
def test_lumina768_strategies_sampled(strategy):
    wl = W.LUMINA768
    _run_and_check(wl, [3], [(3, 5)], _steps(wl, extra=(500,)), all_heads=False, strategy=strategy)


@pytest.mark.parametrize("strategy", STRATEGIES, ids=STRATEGY_IDS)
def test_lumina1024_strategies_sampled(strategy):
    wl = W.LUMINA1024
    _run_and_check(wl, [9], [(9, 1)], _steps(wl), all_heads=False, strategy=strategy)


def test_janus7b_grouped_sampled():
    wl = W.JANUS7B
    _run_and_check(wl, [4], [(4, 9)], _steps(wl), all_heads=False, strategy=B.HEADKV_ATTN_GROUPED)


# ---- grouping and eviction variants: other tau, r_s and grouping points ----

@pytest.mark.parametrize("tau", [0.85, 0.95])
def test_lumina768_tau_sweep(tau):
    # labels, n* and budgets of every head of two layers, retained sets of one
    # slice through the first updates, at another grouping threshold tau
    wl = W.LUMINA768.with_(tau=tau)
    t_g, P = wl.group_threshold - 1, wl.period
    steps = [t_g - 1, t_g, t_g + 1, t_g + P, t_g + 2 * P]
    _run_and_check(wl, [0, 20], [(20, 6)], steps, n_steps=t_g + 2 * P + 1)


@pytest.mark.parametrize("r_s", [(0, 1), (1, 4), (3, 4), (1, 1)], ids=["0", "1/4", "3/4", "1"])
def test_tiny_rs_sweep(r_s):
    # r_s = 0 or 1 leaves one part: plain bottom-M eviction over the history
    wl = W.TINY.with_(r_s=r_s)
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
    torch.cuda.synchronize()
    _check_slice(wl, res, 0, 0, steps)


@pytest.mark.parametrize("r_s", [(0, 1), (1, 1)], ids=["0", "1"])
def test_lumina768_rs_extremes(r_s):
    wl = W.LUMINA768.with_(rho=(1, 4), r_s=r_s)
    _run_and_check(wl, [2], [(2, 4)], _steps(wl), all_heads=False)


@pytest.mark.parametrize("thr", [100, 1200])
def test_lumina768_other_grouping_points(thr):
    # grouping at an earlier or later step (the labels' stability across
    # positions is read from these)
    wl = W.LUMINA768.with_(group_threshold=thr)
    t_g, P = thr - 1, wl.period
    steps = [t_g, t_g + 1, t_g + P]
    _run_and_check(wl, [11], [(11, 1)], steps, n_steps=t_g + P + 1)


# ---- classifier-free-guidance pairs and the LlamaGen-XL shape (d = 64) ----

def test_tiny_cfg_pairs_every_step():
    # row 1 (unconditional) takes row 0's labels: budgets, policies and
    # retained sets follow them
    wl = W.TINY.with_(batch=2, cfg_pairs=True)
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
    torch.cuda.synchronize()
    for b in (0, 1):
        _check_slice(wl, res, 0, b, steps)


def test_llamagen_xl_cfg_sampled():
    wl = W.LLAMAGEN_XL
    _run_and_check(wl, [0, 35], [(0, 0), (35, 255)], _steps(wl, extra=(250,)))


# ---- prefill: causal attention over the conditional tokens (MFMA) ----

@pytest.mark.parametrize("wl", [W.TINY, W.JANUS7B.with_(layers=1), W.LUMINA768.with_(layers=1),
                                W.LLAMAGEN_XL.with_(layers=1, batch=4),
                                W.LUMINA768.with_(layers=1, prefix_len=77, batch=2),
                                W.LUMINA768.with_(layers=1, prefix_len=300, batch=1)],
                         ids=["tiny", "janus", "lumina768", "llamagen", "c77", "c300"])
def test_prefill_attention(wl):
    qc = synth.prefix_q(wl, 0, "cuda")
    kc, vc = synth.prefix_kv(wl, 0, "cuda")
    sess = new_session(wl)
    out = sess.prefill_attn(0, qc, kc, vc)
    torch.cuda.synchronize()
    out = out.cpu().double().numpy()
    qh, kh, vh = qc.cpu(), kc.cpu(), vc.cpu()
    BH = wl.batch * wl.heads
    worst = 0.0
    for i in sorted({0, BH // 3, BH - 1}):
        b, h = divmod(i, wl.heads)
        ref = oracle.prefill_attention(qh[b, h], kh[b, h], vh[b, h])
        err = float(np.abs(out[b, h] - ref).max())
        worst = max(worst, err)
        assert err <= ATOL, (b, h, err)
    _say(f"prefill attention {wl.name} C={wl.prefix_len} d={wl.head_dim}: max err {worst:.2e}")


def test_prefill_attention_then_decode():
    # headkv_prefill_attn leaves the cache as headkv_prefill does
    wl = W.TINY
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    sess.prefill_attn(0, inp.qc[0], inp.kc[0], inp.vc[0])
    out = sess.decode_step(0, 0, inp.q[0][0], inp.k[0][0], inp.v[0][0])
    torch.cuda.synchronize()
    for h in range(wl.heads):
        q, k, v, kc, vc = synth.head_inputs(wl, 0, 0, h)
        ref = oracle.attention(q[0], torch.cat([kc, k[:1]]), torch.cat([vc, v[:1]]))
        assert np.abs(out[0, h].cpu().double().numpy() - ref).max() <= ATOL


@pytest.mark.parametrize("t_end", [200, 300 + 2 * 49 + 5])
def test_decode_attn_layers_matches_per_layer(t_end):
    # one launch for several layers gives the per-layer results: in the
    # full-cache phase (heads of 328 tokens, three-quarter passes) and after
    # two updates
    wl = W.LUMINA768.with_(layers=3)
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    run_generation(sess, inp, steps=t_end)
    t = t_end - 1
    q = [inp.q[l][t] for l in range(3)]
    per = [sess.decode_attn(l, q[l]) for l in range(3)]
    together = [torch.empty_like(p) for p in per]
    B.headkv_decode_attn_layers(sess.h, 0, 3, [x.data_ptr() for x in q],
                                [x.data_ptr() for x in together], sess.stream())
    torch.cuda.synchronize()
    for l in range(3):
        assert float((per[l] - together[l]).abs().max()) <= 1e-5
    ref = oracle.simulate(wl, 1, 4, snap_steps=[t])
    got = together[1][4].cpu().double().numpy()
    for h in range(wl.heads):
        assert np.abs(got[h] - ref["out"][h][t]).max() <= ATOL


# ---- attention-sum eviction scores (variant of Eq. 6) ----

@pytest.mark.parametrize("fused", [True, False])
def test_tiny_attention_sum_scores_every_step(fused):
    wl = W.TINY.with_(score_mode=B.HEADKV_SCORE_ATTN_SUM)
    steps = list(range(wl.num_visual))
    inp = DeviceInputs(wl)
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps, fused=fused)
    torch.cuda.synchronize()
    _check_slice(wl, res, 0, 0, steps)


@pytest.mark.parametrize("wl", [W.LUMINA768.with_(score_mode=1),
                                W.STRESS.with_(score_mode=1, batch=4),
                                W.LUMINA1024.with_(score_mode=1)],
                         ids=["lumina768", "stress_b4", "lumina1024"])
def test_attention_sum_scores_sampled(wl):
    t_g, P = wl.group_threshold - 1, wl.period
    steps = [t_g, t_g + 1, t_g + P, t_g + 3 * P, t_g + 3 * P + 1]
    _run_and_check(wl, [1], [(1, 2)], steps, all_heads=False, n_steps=steps[-1] + 1)

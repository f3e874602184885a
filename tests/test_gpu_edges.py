"""Edge cases of the decode path on small synthetic workloads, every step of
the generation checked against the oracle (bit-exact retained sets, labels, n*
and budgets; attention within 2e-2)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_20600_amd import binding as B, synth, workloads as W
from paper_2605_20600_amd.runner import DeviceInputs, new_session, run_generation
from parity_report import assert_same_retained

pytestmark = pytest.mark.gpu
ATOL = 2e-2


def _run(wl, layer=0, slices=((0, 0),), budgets=None, fused=True, steps=None, **cfg):
    steps = list(range(wl.num_visual)) if steps is None else steps
    inp = DeviceInputs(wl, layers=[layer])
    if budgets is not None:
        inp.override[layer] = torch.as_tensor(np.asarray(budgets, dtype=np.int32).reshape(-1),
                                              device="cuda")
    sess = new_session(wl, **cfg)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps, fused=fused)
    torch.cuda.synchronize()
    H = wl.heads
    worst = 0.0
    for (_, b) in slices:
        ov = None if budgets is None else np.asarray(budgets).reshape(wl.batch, H)[b]
        ref = oracle.simulate(wl, layer, b, snap_steps=steps, budget_override=ov)
        sl = slice(b * H, (b + 1) * H)
        assert np.array_equal(res["is_local"][layer][sl].cpu().numpy(), ref["labels"])
        assert np.array_equal(res["n_star"][layer][sl].cpu().numpy(), ref["n_star"])
        assert np.array_equal(res["budgets"][layer][sl].cpu().numpy(), ref["budgets"])
        masks = [res["snap"][(t, layer)][0][sl].cpu().numpy() for t in steps]
        assert_same_retained(steps, masks, ref, range(H), wl.period, wl.group_threshold - 1,
                             f"{wl.name} b {b}:")
        for i, t in enumerate(steps):
            out = res["out"][(t, layer)][b].cpu().double().numpy()
            for h in range(H):
                err = float(np.abs(out[h] - ref["out"][h][t]).max())
                worst = max(worst, err)
                assert err <= ATOL, (b, h, t, err)
    return res, worst


def test_no_prefix():
    _run(W.TINY.with_(prefix_len=0))


def test_budgets_below_recent_window():
    wl = W.TINY.with_(budget_mode=W.BUDGET_OVERRIDE)
    _run(wl, budgets=[[5, 1, 7, 31]])


def test_update_every_step():
    _run(W.TINY.with_(period=1))


@pytest.mark.parametrize("fused", [True, False])
def test_period_not_dividing_rows(fused):
    _run(W.TINY.with_(period=7, group_threshold=50), fused=fused)


def test_period_longer_than_generation():
    # P > N: the grouping step's update is the only one, and its window of
    # past queries starts at step 0 (the library keeps min(P, N) of them)
    _run(W.TINY.with_(period=300))


@pytest.mark.parametrize("fused", [True, False])
def test_window_longer_than_one_staging_chunk(fused):
    # a window of 100 queries is summed in two chunks of the update's LDS stage
    # (64 + 36 steps), the grouping window in one (steps 0..63)
    _run(W.TINY.with_(period=100, group_threshold=64), fused=fused)


@pytest.mark.parametrize("r_s", [(0, 1), (1, 1), (3, 10), (4, 5)])
def test_stratification_ratio(r_s):
    _run(W.TINY.with_(r_s=r_s), r_s=r_s)


@pytest.mark.parametrize("tau", [0.85, 0.95, 1.0])
def test_grouping_threshold_tau(tau):
    _run(W.TINY.with_(tau=tau), tau=tau)


@pytest.mark.parametrize("thr", [1, 2, 256])
def test_grouping_at_first_and_last_steps(thr):
    _run(W.TINY.with_(group_threshold=thr))


def test_row_end_tokens_odd_grid():
    wl = W.TINY.with_(grid_rows=11, grid_cols=13, row_end=True, period=14, group_threshold=40,
                      heads=6, batch=2)
    _run(wl, slices=((0, 0), (0, 1)))


def test_many_heads_dispatch_order_d64():
    # 8 x 40 = 320 heads per layer: more attention blocks than compute units
    wl = W.TINY.with_(batch=8, heads=40, budget_mode=W.BUDGET_OVERRIDE)
    rng = np.random.default_rng(5)
    bud = rng.integers(1, 257, size=(8, 40))
    _run(wl, budgets=bud, slices=((0, 0), (0, 7)), steps=[0, 63, 64, 65, 100, 200, 255])


def test_few_long_heads_split_d64():
    # 1 x 2 heads of up to 1024 tokens: each head split over several blocks
    wl = W.TINY.with_(heads=2, grid_rows=32, grid_cols=32, period=32, group_threshold=600,
                      budget_mode=W.BUDGET_OVERRIDE)
    _run(wl, budgets=[[1000, 900]], steps=[0, 300, 599, 600, 601, 800, 1023])


# 2 heads of d = 128 that grow to 3,000 tokens before grouping and keep up to
# 3,500 after it: before grouping the layer's chunk table cuts them into
# 128-token chunks (every count from 1 to 24 as they grow: merge trees of up
# to five levels, most of them not full), after it into 512-token chunks (up
# to 8)
DEEP_TREES = W.TINY.with_(heads=2, head_dim=128, grid_rows=64, grid_cols=64, period=64,
                          group_threshold=3000, budget_mode=W.BUDGET_OVERRIDE)
DEEP_TREE_BUDGETS = [[3500, 1800]]
DEEP_TREE_STEPS = [0, 95, 96, 127, 223, 351, 500, 863, 1000, 1500, 2047, 2048, 2998, 2999, 3000,
                   3001, 3063, 3064, 3065, 4095]


def test_deep_merge_trees_d128():
    _run(DEEP_TREES, budgets=DEEP_TREE_BUDGETS, steps=DEEP_TREE_STEPS)


def test_large_logits():
    # amplitudes x4: a planted head's logit for its own position is ~600 nats
    # (exp overflows fp32 past ~88), so every merge of the softmax -- passes,
    # rows, wavefronts, chunks -- must rescale to a common max
    _run(W.TINY.with_(amp_scale=4.0))


def test_large_logits_many_heads_several_passes():
    # the same amplitudes over 320 heads of up to 1056 tokens: one block per
    # head, more blocks than compute units, up to three passes per block
    wl = W.TINY.with_(batch=8, heads=40, grid_rows=32, grid_cols=32, period=32,
                      group_threshold=600, budget_mode=W.BUDGET_OVERRIDE, amp_scale=4.0)
    rng = np.random.default_rng(11)
    bud = rng.integers(1, 1025, size=(8, 40))
    _run(wl, budgets=bud, slices=((0, 0), (0, 7)), steps=[0, 511, 599, 600, 601, 900, 1023])


def test_pass_boundaries_d128():
    # 8 x 32 = 256 heads of d = 128: one 1024-thread block per head.  Before
    # grouping every head caches C + t tokens at step t and attends one more;
    # a launch whose heads need more than one pass takes passes of 512 or 384
    # tokens, whichever loads fewer rows in all, each pass's rows requested
    # while the previous one finishes.  Cached rows at the steps below: 575
    # (one wide pass of 576), 576 and 767 (two of 384: the second with 192 and
    # 383 rows), 768 and 1023 (two of 512), 1024 (three of 384), 1535 (three of
    # 512, the last with 511 rows), 1536 (four of 384, all full)
    wl = W.TINY.with_(batch=8, heads=32, head_dim=128, grid_rows=40, grid_cols=41, period=41,
                      group_threshold=1600)
    C = wl.prefix_len
    rows = (575, 576, 767, 768, 1023, 1024, 1535, 1536)
    steps = [n - C for n in rows] + [1600, 1639]
    _run(wl, slices=((0, 0), (0, 7)), steps=steps)


def test_limits_prefix_capacity_and_length():
    # the documented limits at once: a 2048-token prefix, 16384 visual tokens
    # and heads holding HEADKV_MAX_CAPACITY = 4608 visual tokens (budget 4480 +
    # period 128); heads 0-1 are planted local (sliding window), 2-3 global (STE)
    wl = W.TINY.with_(heads=4, head_dim=128, prefix_len=2048, grid_rows=128, grid_cols=128,
                      period=128, group_threshold=256, budget_mode=W.BUDGET_OVERRIDE)
    N, P, t_g = wl.num_visual, wl.period, wl.group_threshold - 1
    bud = [B.HEADKV_MAX_CAPACITY - P, 256, B.HEADKV_MAX_CAPACITY - P, 256]
    # steps: grouping, the first updates, a global head at full capacity just
    # before an update, the last steps
    k_full = (B.HEADKV_MAX_CAPACITY - P - (t_g + 1)) // P + 2
    steps = sorted({0, t_g - 1, t_g, t_g + 1, t_g + P - 1, t_g + P, t_g + k_full * P - 1,
                    t_g + k_full * P, N // 2, N - 2, N - 1})
    inp = DeviceInputs(wl, layers=[0])
    inp.override[0] = torch.as_tensor(np.asarray(bud, dtype=np.int32), device="cuda")
    sess = new_session(wl)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
    torch.cuda.synchronize()
    ref = oracle.simulate(wl, 0, 0, snap_steps=steps, budget_override=bud, want_out=False)
    assert list(ref["labels"]) == [1, 1, 0, 0]
    assert np.array_equal(res["is_local"][0].cpu().numpy(), ref["labels"])
    assert np.array_equal(res["n_star"][0].cpu().numpy(), ref["n_star"])
    assert np.array_equal(res["budgets"][0].cpu().numpy(), ref["budgets"])
    heads = [synth.head_inputs(wl, 0, 0, h) for h in range(wl.heads)]
    worst, full = 0.0, 0
    for i, t in enumerate(steps):
        mask, count = res["snap"][(t, 0)]
        mask, count = mask.cpu().numpy(), count.cpu().numpy()
        out = res["out"][(t, 0)][0].cpu().double().numpy()
        for h in range(wl.heads):
            assert np.array_equal(mask[h], ref["snaps"][h][i]), (h, t)
            full = max(full, int(count[h]))
            q, k, v, kc, vc = heads[h]
            keep = np.nonzero(mask[h])[0]
            exp = oracle.attention(q[t], torch.cat([kc, k[keep]]), torch.cat([vc, v[keep]]))
            err = float(np.abs(out[h] - exp).max())
            worst = max(worst, err)
            assert err <= ATOL, (h, t, err)
    assert full == B.HEADKV_MAX_CAPACITY - 1  # a head one token short of its capacity
    print(f"limits: bit-exact retained sets, max err {worst:.2e}, largest head {full}", flush=True)


def test_side_streams_two_handles_concurrently():
    # two handles driven from two host threads on two non-default streams at
    # once; each must match the oracle on its own
    from concurrent.futures import ThreadPoolExecutor
    wl = W.TINY
    steps = [0, wl.group_threshold - 1, wl.group_threshold, 100, 200, wl.num_visual - 1]
    inp = DeviceInputs(wl, layers=[0])

    def one(_):
        s = torch.cuda.Stream()
        with torch.cuda.stream(s):
            sess = new_session(wl)
            r = run_generation(sess, inp, out_steps=steps, snap_steps=steps)
            s.synchronize()
        return r

    with ThreadPoolExecutor(max_workers=2) as ex:
        runs = list(ex.map(one, range(2)))
    ref = oracle.simulate(wl, 0, 0, snap_steps=steps)
    for r in runs:
        assert np.array_equal(r["is_local"][0].cpu().numpy(), ref["labels"])
        assert np.array_equal(r["budgets"][0].cpu().numpy(), ref["budgets"])
        for i, t in enumerate(steps):
            mask = r["snap"][(t, 0)][0].cpu().numpy()
            out = r["out"][(t, 0)][0].cpu().double().numpy()
            for h in range(wl.heads):
                assert np.array_equal(mask[h], ref["snaps"][h][i]), (h, t)
                assert float(np.abs(out[h] - ref["out"][h][t]).max()) <= ATOL, (h, t)


def test_wide_pass_d64():
    # 8 x 32 heads of d = 64 in 1024-thread blocks (128 rows): near the end the
    # longest head reads up to 32 + 1031 + 1 tokens, more than one pass of 8
    # tokens per row (1024) and within one of 9 (1152)
    wl = W.TINY.with_(batch=8, heads=32, grid_rows=32, grid_cols=32, period=32,
                      group_threshold=100, budget_mode=W.BUDGET_OVERRIDE)
    rng = np.random.default_rng(11)
    bud = rng.integers(64, 1001, size=(8, 32))
    bud[0, 3] = bud[7, 30] = 1000
    _run(wl, budgets=bud, slices=((0, 0), (0, 7)),
         steps=[99, 100, 500, 990, 1000, 1010, 1022, 1023])


@pytest.mark.parametrize("fused,strategy", [(True, 0), (False, 0), (True, 1)],
                         ids=["fused", "separate", "fused-padded"])
def test_update_and_attention_in_one_launch(fused, strategy):
    # 24 x 24 = 576 heads: the attention runs one 256-thread block per head, so
    # each update step's append, update and attention go out as one launch
    # (fused) or as the separate calls; every step checked, with per-head
    # lengths and with padding + mask
    wl = W.TINY.with_(batch=24, heads=24, period=4)
    _run(wl, slices=((0, 0), (0, 23)), fused=fused, attn_strategy=strategy)

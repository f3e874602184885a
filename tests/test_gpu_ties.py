"""Exact ties on the GPU path, against the oracle.

Seeded random inputs almost never give two equal fp64 scores, so the rules for
equal values would go unexercised.  These tests plant them, the same way on
the inputs of both sides (the edited inputs are built on the CPU and copied to
the device; nothing the oracle reads comes from the library):

  * grouping (Sec. 4, Step 2): a zero query gives every cached token the same
    weight 1/L; with L = 64 and tau = 31/64 the backward mass S(31) equals tau
    exactly, so n* = 31 only if the mass *reaching* tau counts, and with a
    local window of 32 the label then hangs on it too;
  * Stratified Token Eviction (Eqs. 4-6): zero queries over the window before
    one update make every score of that update 0, so every part evicts purely
    by the tie rule (among equal scores the older token leaves); and a key
    copied onto another token at an eviction boundary gives two equal scores
    of which exactly one leaves.

Each case asserts that the oracle itself met the planted tie (a grouping
margin or an eviction-score gap of exactly 0), then compares labels, n*,
budgets and every step's retained set bit-exactly, and attention within 2e-2.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_20600_amd import workloads as W
from paper_2605_20600_amd.runner import DeviceInputs, new_session, run_generation
from parity_report import assert_same_retained

pytestmark = pytest.mark.gpu
ATOL = 2e-2


class _Inputs:
    """The fields of DeviceInputs, copied to another device."""

    def __init__(self, src: DeviceInputs, device: str):
        self.wl, self.layers = src.wl, src.layers
        for name in ("q", "k", "v", "kc", "vc", "qc", "override"):
            setattr(self, name, {l: (None if t is None else t.to(device))
                                 for l, t in getattr(src, name).items()})


def _slice(inp, b):
    """{h: (q, k, v, kc, vc)} of layer 0, batch row b (CPU tensors)."""
    return {h: (inp.q[0][:, b, h], inp.k[0][:, b, h], inp.v[0][:, b, h], inp.kc[0][b, h],
                inp.vc[0][b, h]) for h in range(inp.wl.heads)}


def _compare(wl, inp_cpu, slices, fused=True, **cfg):
    """Runs every step of layer 0 on the GPU from the edited CPU inputs and
    compares each slice with the oracle on the same inputs."""
    steps = list(range(wl.num_visual))
    inp = _Inputs(inp_cpu, "cuda")
    sess = new_session(wl, **cfg)
    res = run_generation(sess, inp, out_steps=steps, snap_steps=steps, fused=fused)
    torch.cuda.synchronize()
    H = wl.heads
    refs = {}
    for b in slices:
        ref = oracle.simulate(wl, 0, b, snap_steps=steps, inputs=_slice(inp_cpu, b))
        sl = slice(b * H, (b + 1) * H)
        assert np.array_equal(res["is_local"][0][sl].cpu().numpy(), ref["labels"]), "labels"
        assert np.array_equal(res["n_star"][0][sl].cpu().numpy(), ref["n_star"]), "n*"
        assert np.array_equal(res["budgets"][0][sl].cpu().numpy(), ref["budgets"]), "budgets"
        masks = [res["snap"][(t, 0)][0][sl].cpu().numpy() for t in steps]
        assert_same_retained(steps, masks, ref, range(H), wl.period, wl.group_threshold - 1,
                             f"{wl.name} b {b}:")
        worst = 0.0
        for t in steps:
            out = res["out"][(t, 0)][b].cpu().double().numpy()
            for h in range(H):
                err = float(np.abs(out[h] - ref["out"][h][t]).max())
                worst = max(worst, err)
                assert err <= ATOL, (b, h, t, err)
        refs[b] = ref
        print(f"{wl.name} {wl.batch}x{wl.heads} b {b}: ties bit-exact, max err {worst:.2e}",
              flush=True)
    return refs


def test_grouping_mass_exactly_tau():
    # C = 32 prefix + 32 visual tokens at grouping: L = 64, a power of two, so
    # every weight of a zero query is exactly 1/64 and S(31) = 31/64 = tau
    wl = W.TINY.with_(group_threshold=32, tau=31 / 64)
    assert wl.prefix_len + wl.group_threshold == 64 and wl.local_window == 32
    t_g = wl.group_threshold - 1
    inp = DeviceInputs(wl, layers=[0], device="cpu")
    tied = (1, 3)  # one planted-local and one planted-global head
    for h in tied:
        inp.q[0][t_g, 0, h] = 0
    refs = _compare(wl, inp, [0], tau=wl.tau)
    ref = refs[0]
    for h in tied:
        # the oracle met the tie: mass equal to tau, hence n* = 31 < 32, local
        assert ref["margin"][h] == 0.0 and ref["n_star"][h] == 31 and ref["labels"][h] == 1, h
        assert ref["mass_window"][h] == wl.tau


def _zero_window_queries(wl, inp, min_step):
    """Zeroes every head's queries over the window of the first update at or
    after min_step (steps t_u - P + 1 .. t_u); returns t_u."""
    t_g, P = wl.group_threshold - 1, wl.period
    t_u = t_g + max(1, -(-(min_step - t_g) // P)) * P
    inp.q[0][t_u - P + 1: t_u + 1] = 0
    return t_u


@pytest.mark.parametrize("batch,heads,period,fused",
                         [(1, 4, 16, True), (1, 4, 16, False), (8, 32, 16, True),
                          (24, 24, 4, True)],
                         ids=["chunked-fused", "chunked-separate", "256heads-update+attn1024",
                              "576heads-update+attn256"])
def test_all_scores_tied_at_one_update(batch, heads, period, fused):
    # every Eq. 6 score of the update is (sum of zero queries) . k = 0: the
    # radix selection reaches its exact threshold key in every evicting part
    # and must take the oldest tokens.  Global heads of rho = 1/2 evict from
    # step 128 on.  256 heads run the update inside the attention kernel in
    # 1024-thread blocks, 576 heads in 256-thread blocks, 4 heads in the
    # separate update kernel
    wl = W.TINY.with_(batch=batch, heads=heads, period=period)
    inp = DeviceInputs(wl, layers=[0], device="cpu")
    t_u = _zero_window_queries(wl, inp, 160)
    slices = sorted({0, batch - 1})
    refs = _compare(wl, inp, slices, fused=fused)
    glob = [(b, h) for b in slices for h in range(heads) if refs[b]["labels"][h] == 0]
    assert glob, "no global head"
    for b, h in glob:
        assert refs[b]["stats"][h]["min_gap"] == 0.0, (b, h, t_u)


def _plant_boundary_tie(wl, inp, b, h, t_u):
    """Copies onto a token kept at the update of step t_u the key of the token
    with the highest score the update evicts, trying kept tokens nearest in
    position first, until the oracle meets an exact tie at an eviction
    boundary.  Returns the pair of positions."""
    P = wl.period
    q, k, v, kc, vc = _slice(inp, b)[h]
    t_g = wl.group_threshold - 1

    def run(kk):
        base = oracle.simulate(wl, 0, b, heads=[h], want_out=False, snap_steps=[t_u - 1, t_u],
                               inputs={**_slice(inp, b), h: (q, kk, v, kc, vc)})
        return base

    base = run(k)
    assert base["labels"][h] == 0, "the head must be global"
    before, after = base["snaps"][h][0].astype(bool), base["snaps"][h][1].astype(bool)
    before[t_u] = True
    gone = np.nonzero(before & ~after)[0]
    assert gone.size > 0, "the update must evict"
    qsum = q[t_u - P + 1: t_u + 1].double().sum(0)
    score = lambda p: float(qsum @ k[p].double())
    a = max(gone.tolist(), key=score)
    recent = set(np.nonzero(after)[0].tolist()[-wl.recent_len:])
    kept = [p for p in np.nonzero(after)[0].tolist() if p not in recent]
    for p in sorted(kept, key=lambda p: abs(p - a))[:24]:
        kk = k.clone()
        kk[p] = k[a]
        if run(kk)["stats"][h]["min_gap"] == 0.0:
            inp.k[0][p, b, h] = k[a]
            return a, p
    raise AssertionError("no kept token gave an exact tie at the boundary")


@pytest.mark.parametrize("batch,heads,fused", [(1, 4, True), (1, 4, False), (8, 32, True)],
                         ids=["chunked-fused", "chunked-separate", "256heads-update+attn1024"])
def test_identical_keys_at_eviction_boundary(batch, heads, fused):
    # two tokens with the same key score the same; at the boundary of the
    # bottom-M selection exactly one of them leaves: the older
    wl = W.TINY.with_(batch=batch, heads=heads)
    inp = DeviceInputs(wl, layers=[0], device="cpu")
    t_g, P = wl.group_threshold - 1, wl.period
    t_u = t_g + 7 * P  # an update at which the global heads of rho = 1/2 evict
    b = batch - 1
    planted = []
    for h in range(heads):
        if oracle.group_layer_row(wl, 0, b)[h] == 0:
            planted.append((h, _plant_boundary_tie(wl, inp, b, h, t_u)))
            if len(planted) == 2:
                break
    refs = _compare(wl, inp, [b], fused=fused)
    for h, pair in planted:
        assert refs[b]["stats"][h]["min_gap"] == 0.0, (h, pair)

"""headkv_decode_attn_noalloc, the entry point for callers that cannot allocate,
against headkv_decode_attn through the C ABI.

Both run the same attention kernels; the allocation-free call keeps the
split-K partial results of a chunked layer (fewer batch x heads than compute
units) in the library's static per-GPU scratch array instead of the handle's
workspace.  Its outputs must equal the existing entry point's bit for bit (the
chunks of a head are merged in the same fixed tree either way), hence also lie within
the 2e-2 parity bar of the oracle.  Two calls in a row, the second on a smaller
layer, check that what the first left in the shared scratch does not leak into
the second.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2605_20600_amd import binding as B, workloads as W
from paper_2605_20600_amd.runner import DeviceInputs, new_session, run_generation
from paper_2605_20600_amd.session import Session, make_config

pytestmark = pytest.mark.gpu
ATOL = 2e-2


def _session_at(wl, steps):
    inp = DeviceInputs(wl, layers=[0])
    sess = new_session(wl)
    run_generation(sess, inp, steps=steps)
    torch.cuda.synchronize()
    return inp, sess


def test_noalloc_equals_decode_attn_two_calls_second_smaller():
    cases = [
        # 4 x 32 = 128 heads of up to ~1230 tokens, chunked (after grouping)
        (W.LUMINA1024.with_(layers=1), 500 + 2 * 65 + 7),
        # 4 heads, chunked, a smaller layer (the scratch keeps the first's data)
        (W.TINY, 150),
    ]
    for i, (wl, steps) in enumerate(cases):
        inp, sess = _session_at(wl, steps)
        t = steps - 1
        q = inp.q[0][t]
        got = torch.full((wl.batch, wl.heads, wl.head_dim), float("nan"), device="cuda")
        sess.decode_attn_noalloc(0, q, got)  # first: before the workspace path runs
        ref = sess.decode_attn(0, q)
        again = torch.full_like(got, float("nan"))
        sess.decode_attn_noalloc(0, q, again)
        torch.cuda.synchronize()
        assert torch.equal(got, ref), (wl.name, float((got - ref).abs().max()))
        assert torch.equal(again, ref), wl.name
        assert float((got - ref).abs().max()) <= ATOL
        print(f"call {i + 1}: {wl.name} {wl.batch}x{wl.heads} heads at step {t}: "
              f"bitwise equal to headkv_decode_attn", flush=True)
        sess.close()


def test_noalloc_on_a_handle_without_workspace():
    # a handle created with a NULL workspace: the chunked attention of the
    # plain entry point refuses (HEADKV_ERR_STATE), the allocation-free one
    # runs it; its outputs follow the oracle through grouping and updates
    wl = W.TINY
    t_g, P = wl.group_threshold - 1, wl.period
    check = [0, t_g - 1, t_g, t_g + 1, t_g + P, t_g + 2 * P + 3, wl.num_visual - 1]
    inp = DeviceInputs(wl, layers=[0])
    sess = Session(make_config(wl), workspace=False)
    sess.prefill(0, inp.kc[0], inp.vc[0])
    outs = {}
    out = torch.empty((wl.batch, wl.heads, wl.head_dim), dtype=torch.float32, device="cuda")
    for t in range(wl.num_visual):
        q, k, v = inp.q[0][t], inp.k[0][t], inp.v[0][t]
        sess.append_and_evict(0, t, q, k, v)
        if t == t_g:
            sess.score_heads(0, q)
            sess.assign_budgets(0, override=inp.override[0])
        if t == 0:
            with pytest.raises(B.HeadKVError) as e:
                sess.decode_attn(0, q, out)
            assert e.value.status == B.HEADKV_ERR_STATE
        sess.decode_attn_noalloc(0, q, out)
        if t in check:
            outs[t] = out.clone()
    torch.cuda.synchronize()
    ref = oracle.simulate(wl, 0, 0, snap_steps=check)
    worst = 0.0
    for t in check:
        got = outs[t][0].cpu().double().numpy()
        for h in range(wl.heads):
            err = float(np.abs(got[h] - ref["out"][h][t]).max())
            worst = max(worst, err)
            assert err <= ATOL, (t, h, err)
    print(f"no-workspace handle: {len(check)} steps within {worst:.2e} of the oracle", flush=True)
    sess.close()

"""Drives one image generation through the C ABI, step by step and layer by
layer, in the order a decoder would: append (+ periodic update), grouping at
step thr-1, attention.  Used by the parity tests, the smoke check and the
benchmark."""
from __future__ import annotations

from typing import Dict, Iterable, List, Optional

import torch

from . import binding as B
from . import synth
from .session import Session, make_config
from .workloads import Workload


class DeviceInputs:
    """All synthetic inputs of a generation, resident on the device.
    q, k, v: per layer bf16 [N][B][H][d]; kc, vc: per layer bf16 [B][H][C][d];
    override: per layer int32 [B][H] or None."""

    def __init__(self, wl: Workload, layers: Optional[List[int]] = None, device: str = "cuda",
                 seed: int = synth.SEED_DATA, chunk_steps: int = 512):
        self.wl = wl
        self.layers = list(range(wl.layers)) if layers is None else list(layers)
        self.q, self.k, self.v, self.kc, self.vc, self.override = {}, {}, {}, {}, {}, {}
        self.qc = {}
        ov = synth.budget_override(wl)
        N = wl.num_visual
        for l in self.layers:
            shape = (N, wl.batch, wl.heads, wl.head_dim)
            q = torch.empty(shape, dtype=torch.bfloat16, device=device)
            k = torch.empty_like(q)
            v = torch.empty_like(q)
            for t0 in range(0, N, chunk_steps):
                t1 = min(N, t0 + chunk_steps)
                q[t0:t1], k[t0:t1], v[t0:t1] = synth.visual_qkv(wl, l, t0, t1, device, seed)
            self.q[l], self.k[l], self.v[l] = q, k, v
            self.kc[l], self.vc[l] = synth.prefix_kv(wl, l, device, seed)
            self.qc[l] = synth.prefix_q(wl, l, device, seed)
            self.override[l] = (None if ov is None else
                                torch.from_numpy(ov[l].reshape(-1).copy()).to(device))

    def nbytes(self) -> int:
        return sum(t.numel() * t.element_size()
                   for d in (self.q, self.k, self.v, self.kc, self.vc, self.qc)
                   for t in d.values())


def run_generation(sess: Session, inp: DeviceInputs, out_steps: Iterable[int] = (),
                   snap_steps: Iterable[int] = (), steps: Optional[int] = None,
                   outs: Optional[Dict[int, torch.Tensor]] = None,
                   label_override: Optional[Dict[int, torch.Tensor]] = None,
                   decode_hook=None, record_layers: Optional[Iterable[int]] = None,
                   fused: bool = True) -> Dict:
    """Runs steps 0..steps-1 (default N) of every layer in `inp.layers`.

    Returns {"out": {(t, l): fp32 [B][H][d]}, "snap": {(t, l): (mask, count)},
    "n_star"/"is_local"/"budgets": {l: tensor}} for the requested steps.
    decode_hook(t, l, launch) may wrap the attention launch (timing).
    fused: use headkv_decode_step (append + update + attention in the fewest
    launches) on every step but the grouping step; else the separate calls."""
    wl = inp.wl
    N = wl.num_visual if steps is None else steps
    t_g = wl.group_threshold - 1
    out_steps, snap_steps = set(out_steps), set(snap_steps)
    rec = set(inp.layers if record_layers is None else record_layers)
    res = {"out": {}, "snap": {}, "n_star": {}, "is_local": {}, "budgets": {}}
    if outs is None:
        outs = {l: torch.empty((wl.batch, wl.heads, wl.head_dim), dtype=torch.float32,
                               device=sess.device) for l in inp.layers}
    for l in inp.layers:
        sess.prefill(l, inp.kc[l], inp.vc[l])
    for t in range(N):
        for l in inp.layers:
            q, k, v = inp.q[l][t], inp.k[l][t], inp.v[l][t]
            if fused and t != t_g:
                launch = (lambda: sess.decode_step(l, t, q, k, v, outs[l]))
            else:
                sess.append_and_evict(l, t, q, k, v)
                if t == t_g:
                    n_star, is_local = sess.score_heads(l, q)
                    lab = None if label_override is None else label_override[l]
                    sess.assign_budgets(l, is_local=lab, override=inp.override[l])
                    res["n_star"][l] = n_star.clone()
                    res["is_local"][l] = (is_local if lab is None else lab).clone()
                    res["budgets"][l] = sess.budgets[l].clone()
                launch = (lambda: sess.decode_attn(l, q, outs[l]))
            if decode_hook is None:
                launch()
            else:
                decode_hook(t, l, launch)
            if t in out_steps and l in rec:
                res["out"][(t, l)] = outs[l].clone()
            if t in snap_steps and l in rec:
                res["snap"][(t, l)] = sess.export_retained(l)
    return res


def new_session(wl: Workload, layers: Optional[int] = None, **kw) -> Session:
    return Session(make_config(wl, layers=layers, **kw))


def run_generation_native(sess: Session, inp: DeviceInputs, outs: Dict[int, torch.Tensor],
                          timing_every: int = 0,
                          label_override: Optional[Dict[int, torch.Tensor]] = None,
                          prefill_out: Optional[Dict[int, torch.Tensor]] = None) -> Dict:
    """The same generation with the step loop in the library (headkv_run_steps):
    steps before and after the grouping step run from one host call each; the
    grouping step uses the separate calls; the prefix goes through the prefill
    attention (headkv_prefill_attn, whose outputs land in `prefill_out` when
    given).  Needs the inputs of every layer of the handle.  label_override: per
    layer [B*H] uint8 labels that replace the grouping's for the budgets and
    updates.  Returns labels, n* and budgets per layer."""
    wl = inp.wl
    L = sess.cfg.num_layers
    assert inp.layers == list(range(L)), "the native loop runs every layer"
    t_g = wl.group_threshold - 1
    N = wl.num_visual
    stride = wl.batch * wl.heads * wl.head_dim
    qp = [inp.q[l].data_ptr() for l in range(L)]
    kp = [inp.k[l].data_ptr() for l in range(L)]
    vp = [inp.v[l].data_ptr() for l in range(L)]
    op = [outs[l].data_ptr() for l in range(L)]
    st = sess.stream()
    res = {"n_star": {}, "is_local": {}, "budgets": {}}
    for l in range(L):
        if wl.prefix_len > 0:
            po = None if prefill_out is None else prefill_out[l]
            sess.prefill_attn(l, inp.qc[l], inp.kc[l], inp.vc[l], po)
        else:
            sess.prefill(l, inp.kc[l], inp.vc[l])
    B.headkv_run_steps(sess.h, 0, t_g, qp, kp, vp, stride, op, timing_every, st)
    for l in range(L):
        q = inp.q[l][t_g]
        sess.append_and_evict(l, t_g, q, inp.k[l][t_g], inp.v[l][t_g])
        n_star, is_local = sess.score_heads(l, q)
        lab = None if label_override is None else label_override[l]
        sess.assign_budgets(l, is_local=lab, override=inp.override[l])
        sess.decode_attn(l, q, outs[l])
        res["n_star"][l], res["is_local"][l] = n_star, (is_local if lab is None else lab)
        res["budgets"][l] = sess.budgets[l]
    B.headkv_run_steps(sess.h, t_g + 1, N, qp, kp, vp, stride, op, timing_every, st)
    return res


def grouping_labels(wl: Workload, inp: DeviceInputs) -> Dict[int, torch.Tensor]:
    """Head labels (1 = local) of every layer when grouping runs at step
    wl.group_threshold - 1: the decode steps before it through the library's
    step loop, then the append and headkv_score_heads.  Returns [B*H] uint8
    per layer."""
    L = wl.layers
    t_g = wl.group_threshold - 1
    sess = new_session(wl)
    outs = {l: torch.empty((wl.batch, wl.heads, wl.head_dim), dtype=torch.float32,
                           device=sess.device) for l in range(L)}
    stride = wl.batch * wl.heads * wl.head_dim
    ptr = lambda d: [d[l].data_ptr() for l in range(L)]
    for l in range(L):
        sess.prefill(l, inp.kc[l], inp.vc[l])
    B.headkv_run_steps(sess.h, 0, t_g, ptr(inp.q), ptr(inp.k), ptr(inp.v), stride, ptr(outs), 0,
                       sess.stream())
    labels = {}
    for l in range(L):
        q = inp.q[l][t_g]
        sess.append_and_evict(l, t_g, q, inp.k[l][t_g], inp.v[l][t_g])
        _, is_local = sess.score_heads(l, q)
        labels[l] = is_local.clone()
    torch.cuda.synchronize()
    sess.close()
    return labels

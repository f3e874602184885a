"""CPU oracle for the head-aware compressed-KV decode path -- TEST INFRASTRUCTURE.

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package.  It wraps the fp64 C library built from `headkv_oracle.c` (see the
header there for the passages each function follows) and shares nothing with
the HIP library except the seeded input generator.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "headkv_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

BUDGET_PAPER, BUDGET_OVERRIDE, BUDGET_TOTAL = 0, 1, 2
SCORE_MEAN_LOGIT, SCORE_ATTN_SUM = 0, 1


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fused multiply-add, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        i = ctypes.c_int
        L.orc_attention.argtypes = [P, P, P, i, i, P]
        L.orc_group_head.argtypes = [P, P, i, i, ctypes.c_double, i, P, P, P, P]
        L.orc_budgets.argtypes = [i, i, P, P, i, i, i, i, i, P]
        L.orc_update.argtypes = [P, P, P, i, P, i, i, i, i, i, i, P, P]
        L.orc_update_ex.argtypes = [P, P, P, i, P, i, i, i, i, i, i, i, P, i, i, P, i, P, P]
        L.orc_run_head.argtypes = [P, P, P, P, P, i, i, i, i, i, i, i, i, i, i,
                                   P, P, i, P, P, i]
        for f in (L.orc_attention, L.orc_group_head, L.orc_budgets, L.orc_update,
                  L.orc_update_ex, L.orc_run_head):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f64(a) -> np.ndarray:
    if isinstance(a, torch.Tensor):
        a = a.detach().cpu().to(torch.float64).numpy()   # bf16 -> f64 is exact
    return np.ascontiguousarray(a, dtype=np.float64)


def _check(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with status {rc}")


def attention(q, K, V) -> np.ndarray:
    """Eq. (1) for one query: q [d], K/V [L][d] -> o [d] (fp64)."""
    q, K, V = _f64(q), _f64(K), _f64(V)
    out = np.empty(q.shape[0], dtype=np.float64)
    _check(lib().orc_attention(_p(q), _p(K), _p(V), K.shape[0], q.shape[0], _p(out)),
           "attention")
    return out


def prefill_attention(qc, kc, vc) -> np.ndarray:
    """Causal attention over the prefix, Eq. (1) token by token: row i attends
    over keys 0..i.  qc, kc, vc: [C][d]; returns fp64 [C][d]."""
    qc, kc, vc = _f64(qc), _f64(kc), _f64(vc)
    return np.stack([attention(qc[i], kc[: i + 1], vc[: i + 1]) for i in range(qc.shape[0])])


def group_head(q, K, tau: float, local_window: int) -> Dict[str, float]:
    """Head grouping of Sec. 4 Step 2 for one head (K in cache order)."""
    q, K = _f64(q), _f64(K)
    ns = np.zeros(1, np.int32)
    loc = np.zeros(1, np.int32)
    mw = np.zeros(1, np.float64)
    mg = np.zeros(1, np.float64)
    _check(lib().orc_group_head(_p(q), _p(K), K.shape[0], q.shape[0], float(tau),
                                int(local_window), _p(ns), _p(loc), _p(mw), _p(mg)),
           "group_head")
    return {"n_star": int(ns[0]), "is_local": int(loc[0]), "mass_window": float(mw[0]),
            "margin": float(mg[0])}


def budgets(mode: int, labels: Sequence[int], N: int, row_len: int, recent_len: int,
            rho=(1, 8), override: Optional[Sequence[int]] = None) -> np.ndarray:
    lab = np.ascontiguousarray(labels, dtype=np.int32)
    ov = None if override is None else np.ascontiguousarray(override, dtype=np.int32)
    out = np.zeros(lab.shape[0], np.int32)
    _check(lib().orc_budgets(int(mode), lab.shape[0], _p(lab), _p(ov), int(N), int(row_len),
                             int(recent_len), int(rho[0]), int(rho[1]), _p(out)), "budgets")
    return out


def update(ret: Sequence[int], Kvis, qsum, budget: int, is_local: bool, recent_len: int,
           r_s=(1, 2), u: int = 0, score_mode: int = SCORE_MEAN_LOGIT, Qwin=None,
           first_step: int = 0, Kc=None):
    """One periodic update (Eqs. 2-6).  Returns (new retained positions, gap).
    score_mode SCORE_ATTN_SUM scores with the window queries Qwin (steps
    first_step ..) over the prefix keys Kc and the retained keys."""
    r = np.zeros(max(len(ret), 1), np.int32)
    r[: len(ret)] = np.asarray(ret, dtype=np.int32)
    n = np.array([len(ret)], np.int32)
    Kv = _f64(Kvis)
    qs = None if qsum is None else _f64(qsum)
    Qw = None if Qwin is None else _f64(Qwin)
    Kc_ = None if Kc is None else _f64(Kc)
    ev = np.zeros(1, np.int32)
    gap = np.zeros(1, np.float64)
    _check(lib().orc_update_ex(_p(r), _p(n), _p(Kv), Kv.shape[1], _p(qs), int(budget),
                               int(bool(is_local)), int(recent_len), int(r_s[0]), int(r_s[1]),
                               int(u), int(score_mode), _p(Qw), 0 if Qw is None else Qw.shape[0],
                               int(first_step), _p(Kc_), 0 if Kc_ is None else Kc_.shape[0],
                               _p(ev), _p(gap)), "update")
    return r[: n[0]].copy(), float(gap[0])


def run_head(q, k, v, kc, vc, t_g: int, P: int, is_local: bool, budget: int,
             recent_len: int, r_s=(1, 2), want_out: bool = True,
             snap_steps: Sequence[int] = (), score_mode: int = SCORE_MEAN_LOGIT):
    """A whole generation of one head; returns (out [N][d] or None, snaps, stats)."""
    q, k, v, kc, vc = _f64(q), _f64(k), _f64(v), _f64(kc), _f64(vc)
    N, d = q.shape
    C = kc.shape[0]
    out = np.empty((N, d), np.float64) if want_out else None
    ss = np.ascontiguousarray(snap_steps, dtype=np.int32)
    masks = np.zeros((max(len(ss), 1), N), np.uint8)
    stats = np.zeros(4, np.float64)
    _check(lib().orc_run_head(_p(q), _p(k), _p(v), _p(kc), _p(vc), C, N, d, int(t_g), int(P),
                              int(bool(is_local)), int(budget), int(recent_len), int(r_s[0]),
                              int(r_s[1]), _p(out), _p(ss) if len(ss) else None, len(ss),
                              _p(masks) if len(ss) else None, _p(stats), int(score_mode)),
           "run_head")
    return out, masks[: len(ss)], {"updates": int(stats[0]), "evicted": int(stats[1]),
                                    "min_gap": float(stats[2])}


def simulate(wl, layer: int, b: int, heads: Optional[List[int]] = None,
             want_out: bool = True, snap_steps: Sequence[int] = (),
             seed: Optional[int] = None, label_override=None, budget_override=None,
             inputs: Optional[Dict] = None) -> Dict:
    """The whole compressed decode of one (layer, b) slice of a workload.

    Grouping runs for every head of the slice (budgets of the layer-total mode
    depend on all labels), then each requested head is run through the
    generation.  Inputs come from the shared seeded generator, or from
    `inputs` ({h: (q, k, v, kc, vc)} CPU tensors of every head of the slice,
    for tests that plant values the generator does not draw).  With
    wl.cfg_pairs the row's budgets and update policies follow the labels of
    its pair's conditional row (b rounded down to even); "labels" and
    "n_star" stay the row's own grouping result."""
    from paper_2605_20600_amd import synth
    kw = {} if seed is None else {"seed": seed}
    H = wl.heads
    heads = list(range(H)) if heads is None else list(heads)
    t_g = wl.group_threshold - 1
    labels = np.zeros(H, np.int32)
    n_star = np.zeros(H, np.int32)
    margins = np.zeros(H, np.float64)
    mass = np.zeros(H, np.float64)
    given = inputs
    inputs = {}
    for h in range(H):
        q, k, v, kc, vc = (synth.head_inputs(wl, layer, b, h, **kw) if given is None
                           else given[h])
        inputs[h] = (q, k, v, kc, vc)
        K = torch.cat([kc, k[: t_g + 1]], dim=0)
        g = group_head(q[t_g], K, wl.tau, wl.local_window)
        labels[h], n_star[h], margins[h], mass[h] = (g["is_local"], g["n_star"],
                                                     g["margin"], g["mass_window"])
    used = labels
    if label_override is not None:
        labels = used = np.asarray(label_override, dtype=np.int32)
    elif getattr(wl, "cfg_pairs", False) and b % 2 == 1:
        used = group_layer_row(wl, layer, b - 1, **kw)
    if budget_override is not None:
        ov_slice = np.asarray(budget_override, dtype=np.int32)
    else:
        ov = synth.budget_override(wl)
        ov_slice = None if ov is None else ov[layer, b]
    bud = budgets(wl.budget_mode, used, wl.num_visual, wl.row_len, wl.recent_len,
                  wl.rho, ov_slice)
    res = {"labels": labels, "n_star": n_star, "margin": margins, "mass_window": mass,
           "budgets": bud, "labels_used": used, "out": {}, "snaps": {}, "stats": {}}
    def one(h):
        q, k, v, kc, vc = inputs[h]
        return h, run_head(q, k, v, kc, vc, t_g, wl.period, bool(used[h]), int(bud[h]),
                           wl.recent_len, wl.r_s, want_out, snap_steps,
                           getattr(wl, "score_mode", SCORE_MEAN_LOGIT))

    # heads are independent; the C code runs without the GIL
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(max_workers=max(1, min(16, os.cpu_count() or 1))) as ex:
        for h, (out, snaps, st) in ex.map(one, heads):
            res["out"][h] = out
            res["snaps"][h] = snaps
            res["stats"][h] = st
    return res


def group_layer_row(wl, layer: int, b: int, seed: Optional[int] = None) -> np.ndarray:
    """Labels of every head of one (layer, batch row): int32 [H]."""
    from paper_2605_20600_amd import synth
    kw = {} if seed is None else {"seed": seed}
    t_g = wl.group_threshold - 1
    lab = np.zeros(wl.heads, np.int32)
    for h in range(wl.heads):
        q, k, _, kc, _ = synth.head_inputs(wl, layer, b, h, **kw)
        lab[h] = group_head(q[t_g], torch.cat([kc, k[: t_g + 1]], dim=0), wl.tau,
                            wl.local_window)["is_local"]
    return lab


def group_layer(wl, layer: int, seed: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Grouping and budgets for every (b, h) of one layer: arrays [B][H].  With
    wl.cfg_pairs, row 2i+1's budgets follow row 2i's labels."""
    from paper_2605_20600_amd import synth
    kw = {} if seed is None else {"seed": seed}
    t_g = wl.group_threshold - 1
    q, k, _ = synth.visual_qkv(wl, layer, 0, t_g + 1, "cpu", **kw)       # [T][B][H][d]
    kc, _ = synth.prefix_kv(wl, layer, "cpu", **kw)                     # [B][H][C][d]
    B, H = wl.batch, wl.heads
    out = {k_: np.zeros((B, H), dt) for k_, dt in (("labels", np.int32), ("n_star", np.int32),
                                                   ("margin", np.float64),
                                                   ("mass_window", np.float64),
                                                   ("budgets", np.int32))}
    ov = synth.budget_override(wl)
    for b in range(B):
        for h in range(H):
            K = torch.cat([kc[b, h], k[:, b, h]], dim=0)
            g = group_head(q[t_g, b, h], K, wl.tau, wl.local_window)
            out["labels"][b, h], out["n_star"][b, h] = g["is_local"], g["n_star"]
            out["margin"][b, h], out["mass_window"][b, h] = g["margin"], g["mass_window"]
    for b in range(B):
        src = b - (b % 2) if getattr(wl, "cfg_pairs", False) else b
        out["budgets"][b] = budgets(wl.budget_mode, out["labels"][src], wl.num_visual, wl.row_len,
                                    wl.recent_len, wl.rho, None if ov is None else ov[layer, b])
    return out

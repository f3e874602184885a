"""Comparison of GPU retained sets with the oracle's, step by step, that names
the first divergent step instead of only asserting.

A retained set that differs at one update changes every later step, so the
report gives the earliest (step, head) among the compared ones, the positions
only one side keeps, and the oracle's margins for that head: its smallest gap
between the last evicted and the first kept eviction score over all updates,
and its grouping margin (distance of the backward attention mass to tau).  A
margin near zero points at a near-tie that the two sides may order
differently; a large one at a plain mistake.
"""
from __future__ import annotations

from typing import Sequence

import numpy as np


def first_divergence(steps: Sequence[int], gpu_masks, ref, heads: Sequence[int], period: int,
                     t_g: int, where: str = ""):
    """gpu_masks[i]: [H][N] uint8 retained masks of step steps[i] (numpy);
    ref: oracle.simulate's result for the same slice and steps.  Returns None
    if every mask agrees, else a message describing the first divergence."""
    order = sorted(range(len(steps)), key=lambda i: steps[i])
    for i in order:
        t = steps[i]
        for h in heads:
            got = np.asarray(gpu_masks[i][h]).astype(bool)
            exp = np.asarray(ref["snaps"][h][i]).astype(bool)
            if np.array_equal(got, exp):
                continue
            only_gpu = np.nonzero(got & ~exp)[0].tolist()
            only_orc = np.nonzero(exp & ~got)[0].tolist()
            upd = t >= t_g and (t - t_g) % period == 0
            prev = [steps[j] for j in order if steps[j] < t]
            return (f"{where} first divergent step {t} (update step: {upd}; last agreeing "
                    f"compared step: {prev[-1] if prev else None}), head {h}: "
                    f"kept only by the GPU {only_gpu[:16]}, only by the oracle {only_orc[:16]}; "
                    f"oracle margins for this head: min eviction-score gap "
                    f"{ref['stats'][h]['min_gap']:.3e}, grouping margin "
                    f"{ref['margin'][h]:.3e} (label {int(ref['labels'][h])}, "
                    f"n* {int(ref['n_star'][h])})")
    return None


def assert_same_retained(steps, gpu_masks, ref, heads, period, t_g, where=""):
    msg = first_divergence(steps, gpu_masks, ref, heads, period, t_g, where)
    assert msg is None, msg

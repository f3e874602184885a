"""Workload shapes for the synthetic compressed-KV decode benchmarks.

Plain data only: every field is a hyper-parameter or a shape, never a value the
method derives (budgets, labels and retained sets are computed by the kernels
and, independently, by the CPU oracle).

Hyper-parameters of the method and where they come from:
  * tau = 0.9 -- attention-mass threshold of head grouping (Sec. 4, Step 2).
  * r_s = 1/2 -- stratification ratio of Stratified Token Eviction (Eq. 5).
  * rho -- budget ratio of global heads, B = rho*N (Sec. 5.1, Implementation
    Details; the B column of the efficiency table).
  * w = two image rows -- recent window (Sec. 5.1, Implementation Details).
  * thr -- visual-token count at which heads are grouped: 100 for Janus-Pro
    and LlamaGen,
    300 for Lumina-mGPT-768, 500 for Lumina-mGPT-1024 (Appendix, More
    Implementation Details).
  * P -- update period of the efficient cache update (Sec. 4, Efficient Cache
    Update); the paper gives no value, one image row is used.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

BUDGET_PAPER = 0     # local heads keep w, global heads keep floor(rho*N)
BUDGET_OVERRIDE = 1  # per-head budgets supplied by the caller
BUDGET_TOTAL = 2     # the layer keeps floor(rho*N)*H in total, split by label


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    layers: int
    heads: int
    head_dim: int
    prefix_len: int            # C, conditional (text) tokens
    grid_rows: int             # image rows
    grid_cols: int             # image tokens per row (without row-end token)
    row_end: bool              # one extra row-end token per row
    period: int                # P
    group_threshold: int       # thr; grouping runs when thr visual tokens are cached
    rho: Tuple[int, int]       # (num, den)
    budget_mode: int
    amp_mode: str              # "tiny", "janus" or "lumina"
    v_positional: bool = False  # add the positional term to V as well
    override: Optional[str] = None  # None, "rows_1_16" or "loguniform_64_1024"
    r_s: Tuple[int, int] = (1, 2)
    tau: float = 0.9
    cfg_pairs: bool = False    # rows 2i / 2i+1: cond / uncond of one guidance pair
    score_mode: int = 0        # 0: Eq. 6 mean logit; 1: summed window attention weights
    amp_scale: float = 1.0     # factor on every positional amplitude (larger logits)

    @property
    def row_len(self) -> int:          # R, including the row-end token
        return self.grid_cols + (1 if self.row_end else 0)

    @property
    def num_visual(self) -> int:       # N
        return self.grid_rows * self.row_len

    @property
    def recent_len(self) -> int:       # w = two rows
        return 2 * self.row_len

    @property
    def local_window(self) -> int:     # W_loc, a head is local iff n* < W_loc
        return self.recent_len

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


TINY = Workload(
    name="tiny", batch=1, layers=1, heads=4, head_dim=64, prefix_len=32,
    grid_rows=16, grid_cols=16, row_end=False, period=16, group_threshold=64,
    rho=(1, 2), budget_mode=BUDGET_PAPER, amp_mode="tiny", v_positional=True)

JANUS7B = Workload(
    name="janus_pro_7b", batch=16, layers=30, heads=32, head_dim=128,
    prefix_len=64, grid_rows=24, grid_cols=24, row_end=False, period=24,
    group_threshold=100, rho=(1, 4), budget_mode=BUDGET_TOTAL, amp_mode="janus")

LUMINA768 = Workload(
    name="lumina_mgpt_768", batch=8, layers=32, heads=32, head_dim=128,
    prefix_len=128, grid_rows=48, grid_cols=48, row_end=True, period=49,
    group_threshold=300, rho=(1, 8), budget_mode=BUDGET_PAPER, amp_mode="lumina")

LUMINA1024 = Workload(
    name="lumina_mgpt_1024", batch=4, layers=32, heads=32, head_dim=128,
    prefix_len=128, grid_rows=64, grid_cols=64, row_end=True, period=65,
    group_threshold=500, rho=(1, 8), budget_mode=BUDGET_OVERRIDE,
    amp_mode="lumina", override="rows_1_16")

STRESS = Workload(
    name="stress_768_b64_p1", batch=64, layers=32, heads=32, head_dim=128,
    prefix_len=128, grid_rows=48, grid_cols=48, row_end=True, period=1,
    group_threshold=300, rho=(1, 8), budget_mode=BUDGET_OVERRIDE,
    amp_mode="lumina", override="loguniform_64_1024")

# LlamaGen-XL (class-conditional, 36 layers, 20 heads of 64, one class token)
# at 384 px: a 24 x 24 grid, 128 images with classifier-free guidance = 256
# sequences in 128 cond/uncond pairs that share their head labels.
LLAMAGEN_XL = Workload(
    name="llamagen_xl", batch=256, layers=36, heads=20, head_dim=64, prefix_len=1,
    grid_rows=24, grid_cols=24, row_end=False, period=24, group_threshold=100,
    rho=(1, 4), budget_mode=BUDGET_PAPER, amp_mode="lumina", cfg_pairs=True)

ALL = {w.name: w for w in (TINY, JANUS7B, LUMINA768, LUMINA1024, STRESS, LLAMAGEN_XL)}

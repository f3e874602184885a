"""A cache session: torch-allocated device buffers for one handle of the C ABI.

PyTorch supplies device memory and the stream; every computation is a call
into libheadkv.so through the binding.
"""
from __future__ import annotations

from typing import List, Optional, Tuple

import torch

from . import binding as B
from .workloads import Workload


def make_config(wl: Workload, rho=None, budget_mode=None, r_s=None, tau=None,
                layers: Optional[int] = None, attn_strategy: int = B.HEADKV_ATTN_VARLEN
                ) -> B.HeadKVConfig:
    rho = wl.rho if rho is None else rho
    r_s = wl.r_s if r_s is None else r_s
    return B.HeadKVConfig(
        batch=wl.batch, num_layers=wl.layers if layers is None else layers,
        num_heads=wl.heads, head_dim=wl.head_dim, prefix_len=wl.prefix_len,
        row_len=wl.row_len, num_visual=wl.num_visual, recent_len=wl.recent_len,
        local_window=wl.local_window, period=wl.period,
        group_threshold=wl.group_threshold,
        budget_mode=wl.budget_mode if budget_mode is None else budget_mode,
        rho_num=rho[0], rho_den=rho[1], rs_num=r_s[0], rs_den=r_s[1],
        attn_strategy=attn_strategy, score_mode=wl.score_mode, cfg_pairs=1 if wl.cfg_pairs else 0,
        tau=wl.tau if tau is None else tau)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


class Session:
    """Owns the device buffers of one handle (dense per-layer caches, metadata,
    workspace, and the per-head segment buffers allocated at grouping)."""

    def __init__(self, cfg: B.HeadKVConfig, device: str = "cuda", workspace: bool = True):
        """workspace=False creates the handle without a workspace (chunked
        attention then goes through headkv_decode_attn_noalloc)."""
        self.cfg = cfg
        self.device = device
        dense_b, meta_b, ws_b = B.headkv_plan(cfg)
        L = cfg.num_layers
        self.dense: List[torch.Tensor] = [torch.empty(dense_b, dtype=torch.uint8, device=device)
                                          for _ in range(L)]
        self.meta: List[torch.Tensor] = [torch.zeros(meta_b, dtype=torch.uint8, device=device)
                                         for _ in range(L)]
        self.ws = (torch.empty(max(ws_b, 256), dtype=torch.uint8, device=device) if workspace
                   else None)
        self.ragged: List[Optional[torch.Tensor]] = [None] * L
        self.h = B.headkv_create(cfg, [t.data_ptr() for t in self.dense],
                                 [t.data_ptr() for t in self.meta],
                                 None if self.ws is None else self.ws.data_ptr())
        BH = cfg.batch * cfg.num_heads
        self.n_star = [torch.zeros(BH, dtype=torch.int32, device=device) for _ in range(L)]
        self.is_local = [torch.zeros(BH, dtype=torch.uint8, device=device) for _ in range(L)]
        self.budgets = [torch.zeros(BH, dtype=torch.int32, device=device) for _ in range(L)]

    @staticmethod
    def stream() -> int:
        return torch.cuda.current_stream().cuda_stream

    def close(self):
        if self.h:
            B.headkv_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- the protocol -----------------------------------------------------
    def prefill(self, layer: int, k_c: Optional[torch.Tensor], v_c: Optional[torch.Tensor]):
        B.headkv_prefill(self.h, layer, _ptr(k_c), _ptr(v_c), self.stream())

    def prefill_attn(self, layer: int, q_c, k_c, v_c, out: Optional[torch.Tensor] = None):
        if out is None:
            out = torch.empty(q_c.shape, dtype=torch.float32, device=self.device)
        B.headkv_prefill_attn(self.h, layer, q_c.data_ptr(), k_c.data_ptr(), v_c.data_ptr(),
                              out.data_ptr(), self.stream())
        return out

    def append_and_evict(self, layer: int, step: int, q, k, v):
        B.headkv_append_and_evict(self.h, layer, step, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                  self.stream())

    def score_heads(self, layer: int, q) -> Tuple[torch.Tensor, torch.Tensor]:
        B.headkv_score_heads(self.h, layer, q.data_ptr(), self.n_star[layer].data_ptr(),
                             self.is_local[layer].data_ptr(), self.stream())
        return self.n_star[layer], self.is_local[layer]

    def assign_budgets(self, layer: int, is_local: Optional[torch.Tensor] = None,
                       override: Optional[torch.Tensor] = None) -> torch.Tensor:
        lab = self.is_local[layer] if is_local is None else is_local
        ov = None if override is None else override.data_ptr()
        st, need = B.headkv_assign_budgets(self.h, layer, lab.data_ptr(), ov,
                                           self.budgets[layer].data_ptr(), None, 0, self.stream())
        assert st == B.HEADKV_ERR_CAPACITY
        buf = self.ragged[layer]
        if buf is None or buf.numel() < need:
            buf = torch.empty(max(need, 256), dtype=torch.uint8, device=self.device)
        st, _ = B.headkv_assign_budgets(self.h, layer, lab.data_ptr(), ov,
                                        self.budgets[layer].data_ptr(), buf.data_ptr(),
                                        buf.numel(), self.stream())
        if st != B.HEADKV_OK:
            raise B.HeadKVError(st, "headkv_assign_budgets", B.headkv_last_error())
        self.ragged[layer] = buf
        return self.budgets[layer]

    def decode_attn(self, layer: int, q, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=self.device)
        B.headkv_decode_attn(self.h, layer, q.data_ptr(), out.data_ptr(), self.stream())
        return out

    def decode_attn_noalloc(self, layer: int, q, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=self.device)
        B.headkv_decode_attn_noalloc(self.h, layer, q.data_ptr(), out.data_ptr(), self.stream())
        return out

    def decode_step(self, layer: int, step: int, q, k, v,
                    out: Optional[torch.Tensor] = None) -> torch.Tensor:
        if out is None:
            out = torch.empty(q.shape, dtype=torch.float32, device=self.device)
        B.headkv_decode_step(self.h, layer, step, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                             out.data_ptr(), self.stream())
        return out

    def export_retained(self, layer: int) -> Tuple[torch.Tensor, torch.Tensor]:
        BH = self.cfg.batch * self.cfg.num_heads
        mask = torch.empty((BH, self.cfg.num_visual), dtype=torch.uint8, device=self.device)
        count = torch.empty(BH, dtype=torch.int32, device=self.device)
        B.headkv_export_retained(self.h, layer, mask.data_ptr(), count.data_ptr(), self.stream())
        return mask, count

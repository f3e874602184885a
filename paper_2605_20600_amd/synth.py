"""Seeded synthetic decode inputs (q, k, v per step, layer, batch row and head).

This module holds no arithmetic of the compression method: it only draws the
inputs, and it draws them bit-identically on the CPU and on the GPU, so that the
CPU oracle and the HIP kernels can be fed the same bf16 values without either
side producing the other's inputs.

How the values are made (all integer hashing plus IEEE fp32 mul/add):
  * noise: a counter-based 32-bit hash of (seed, tensor, layer, step, b, h, dim)
    picks one of 2^16 quantiles of N(0,1); the quantile table is built once in
    fp64 and stored as fp32, so no transcendental is evaluated per element;
  * positional term: a 2-D sinusoid p(r, c) of the visual token's grid cell
    (row r, column c; the row-end token sits in column `grid_cols`); the first
    d/2 dims encode the row, the last d/2 the column, as (sin, cos) pairs with
    frequencies base^(-j/(d/4)); conditional (prefix) tokens carry no term;
  * q = bf16(noise_q + A*p), k = bf16(noise_k + A*p), v = bf16(noise_v)
    (+ A*p when the workload asks for it); A is a per (layer, b, h) amplitude:
    A = 3 plants a locality-biased head, A = 0 a head with no positional bias;
  * every fp32 operation is a separate elementwise mul or add (never fused), and
    the fp32 -> bf16 conversion rounds to nearest even on both devices.
"""
from __future__ import annotations

import functools
import math
from typing import Optional, Tuple

import numpy as np
import torch

from .workloads import Workload

SEED_DATA = 2605
SEED_AMP = 2606
SEED_BUDGET = 2607
POS_BASE = 10.0

T_Q, T_K, T_V, T_KC, T_VC, T_QC = 0, 1, 2, 3, 4, 5
_M32 = 0xFFFFFFFF


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2^32 for int64 x in [0, 2^32) without int64 overflow."""
    lo = x & 0xFFFF
    hi = x >> 16
    return (lo * c + (((hi * c) & 0xFFFF) << 16)) & _M32


def _mix32(x: torch.Tensor) -> torch.Tensor:
    """A bijective 32-bit integer mixer (xorshift-multiply, lowbias32 constants)."""
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


def hash_index(idx: torch.Tensor, seed: int) -> torch.Tensor:
    """32-bit hash of a non-negative int64 counter (< 2^62) under `seed`."""
    lo = idx & _M32
    hi = idx >> 32
    h = _mix32((hi + (seed * 0x9E3779B9)) & _M32)
    return _mix32(lo ^ h)


@functools.lru_cache(maxsize=None)
def normal_table_np() -> np.ndarray:
    """N(0,1) quantiles at (i + 0.5) / 2^16, computed in fp64, stored as fp32."""
    from scipy.special import ndtri
    u = (np.arange(1 << 16, dtype=np.float64) + 0.5) / float(1 << 16)
    return ndtri(u).astype(np.float32)


@functools.lru_cache(maxsize=None)
def _normal_table(device: str) -> torch.Tensor:
    return torch.from_numpy(normal_table_np()).to(device)


@functools.lru_cache(maxsize=None)
def positional_table_np(rows: int, row_len: int, d: int, base: float = POS_BASE) -> np.ndarray:
    """p(r, c) for every visual token in raster order: float32 [rows*row_len][d]."""
    assert d % 4 == 0
    q = d // 4
    omega = base ** (-np.arange(q, dtype=np.float64) / q)
    t = np.arange(rows * row_len)
    r = (t // row_len).astype(np.float64)
    c = (t % row_len).astype(np.float64)
    p = np.empty((t.size, d), dtype=np.float64)
    p[:, 0:d // 2:2] = np.sin(r[:, None] * omega[None, :])
    p[:, 1:d // 2:2] = np.cos(r[:, None] * omega[None, :])
    p[:, d // 2::2] = np.sin(c[:, None] * omega[None, :])
    p[:, d // 2 + 1::2] = np.cos(c[:, None] * omega[None, :])
    return p.astype(np.float32)


@functools.lru_cache(maxsize=None)
def _positional_table(rows: int, row_len: int, d: int, device: str) -> torch.Tensor:
    return torch.from_numpy(positional_table_np(rows, row_len, d)).to(device)


def _small_hash(seed: int, *ids: int, dims: Tuple[int, ...]) -> torch.Tensor:
    """Hash of a small index grid (CPU), used for per-head tables."""
    n = int(np.prod(dims))
    idx = torch.arange(n, dtype=torch.int64)
    return hash_index(idx, seed).reshape(dims)


@functools.lru_cache(maxsize=None)
def amplitudes(wl: Workload, seed: int = SEED_AMP) -> np.ndarray:
    """Positional amplitude A per (layer, b, h): float32 [L][B][H]."""
    L, B, H = wl.layers, wl.batch, wl.heads
    amp = np.zeros((L, B, H), dtype=np.float32)
    if wl.amp_mode == "tiny":
        amp[:, :, : H // 2] = 3.0
    elif wl.amp_mode == "janus":
        hv = _small_hash(seed, dims=(L, B, H)).numpy()
        amp[...] = np.array([0.0, 1.5, 3.0], dtype=np.float32)[(hv >> 8) % 3]
    elif wl.amp_mode == "lumina":
        n_planted = (13 * H + 16) // 32      # 13 of 32 heads (40.6 %)
        hv = _small_hash(seed, dims=(L, B, H)).numpy()
        order = np.argsort(hv, axis=-1, kind="stable")
        chosen = order[..., :n_planted]
        np.put_along_axis(amp, chosen, np.float32(3.0), axis=-1)
    else:
        raise ValueError(wl.amp_mode)
    if wl.amp_scale != 1.0:
        amp *= np.float32(wl.amp_scale)
    return amp


@functools.lru_cache(maxsize=None)
def budget_override(wl: Workload, seed: int = SEED_BUDGET) -> Optional[np.ndarray]:
    """Per-head caller budgets (int32 [L][B][H]) for the override workloads."""
    if wl.override is None:
        return None
    hv = _small_hash(seed, dims=(wl.layers, wl.batch, wl.heads)).numpy().astype(np.float64)
    if wl.override == "rows_1_16":
        rows = 1 + (hv.astype(np.int64) >> 4) % 16
        return (rows * wl.row_len).astype(np.int32)
    if wl.override == "loguniform_64_1024":
        u = (hv + 0.5) / 4294967296.0
        b = np.exp(math.log(64.0) + u * (math.log(1024.0) - math.log(64.0)))
        return np.rint(b).astype(np.int32)
    raise ValueError(wl.override)


def _noise(wl: Workload, tensor: int, layer: int, t: torch.Tensor, b: torch.Tensor,
           h: torch.Tensor, seed: int, device: str) -> torch.Tensor:
    """fp32 N(0,1) draws on the grid t x b x h x dim (broadcast index tensors)."""
    d = wl.head_dim
    tmax = wl.num_visual + wl.prefix_len
    i = torch.arange(d, dtype=torch.int64, device=device)
    base = (tensor * wl.layers + layer) * tmax
    idx = ((((base + t) * wl.batch + b) * wl.heads + h) * d + i)
    hv = hash_index(idx, seed)
    return _normal_table(device)[hv >> 16]


def _visual(wl: Workload, layer: int, t: torch.Tensor, b: torch.Tensor, h: torch.Tensor,
            seed: int, device: str) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    amp_all = torch.from_numpy(amplitudes(wl)[layer]).to(device)          # [B][H]
    pos = _positional_table(wl.grid_rows, wl.row_len, wl.head_dim, device)
    p = pos[t.reshape(-1)].reshape(-1, 1, 1, wl.head_dim)                 # [T,1,1,d]
    a = amp_all[b[..., 0], h[..., 0]].unsqueeze(-1)                         # [1,B,H,1]
    ap = a * p                                                             # fp32 mul
    out = []
    for tensor in (T_Q, T_K, T_V):
        n = _noise(wl, tensor, layer, t, b, h, seed, device)
        if tensor != T_V or wl.v_positional:
            n = n + ap                                                     # fp32 add
        out.append(n.to(torch.bfloat16))
    return out[0], out[1], out[2]


def _grid(t0: int, t1: int, bs, hs, device: str):
    t = torch.arange(t0, t1, dtype=torch.int64, device=device).reshape(-1, 1, 1, 1)
    b = torch.as_tensor(bs, dtype=torch.int64, device=device).reshape(1, -1, 1, 1)
    h = torch.as_tensor(hs, dtype=torch.int64, device=device).reshape(1, 1, -1, 1)
    return t, b, h


def visual_qkv(wl: Workload, layer: int, t0: int, t1: int, device: str = "cpu",
               seed: int = SEED_DATA) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """q, k, v of visual steps [t0, t1) for every (b, h): bf16 [t1-t0][B][H][d]."""
    t, b, h = _grid(t0, t1, range(wl.batch), range(wl.heads), device)
    return _visual(wl, layer, t, b, h, seed, device)


def prefix_kv(wl: Workload, layer: int, device: str = "cpu",
              seed: int = SEED_DATA) -> Tuple[torch.Tensor, torch.Tensor]:
    """Conditional-token keys and values: bf16 [B][H][C][d]."""
    t, b, h = _grid(0, wl.prefix_len, range(wl.batch), range(wl.heads), device)
    t = t + wl.num_visual
    kc = _noise(wl, T_KC, layer, t, b, h, seed, device).to(torch.bfloat16)
    vc = _noise(wl, T_VC, layer, t, b, h, seed, device).to(torch.bfloat16)
    return kc.permute(1, 2, 0, 3).contiguous(), vc.permute(1, 2, 0, 3).contiguous()


def prefix_q(wl: Workload, layer: int, device: str = "cpu",
             seed: int = SEED_DATA) -> torch.Tensor:
    """Conditional-token queries (for the prefill attention): bf16 [B][H][C][d]."""
    t, b, h = _grid(0, wl.prefix_len, range(wl.batch), range(wl.heads), device)
    t = t + wl.num_visual
    qc = _noise(wl, T_QC, layer, t, b, h, seed, device).to(torch.bfloat16)
    return qc.permute(1, 2, 0, 3).contiguous()


def head_inputs(wl: Workload, layer: int, b: int, h: int, seed: int = SEED_DATA):
    """All inputs of one (layer, b, h) head on the CPU, as bf16 tensors:
    q, k, v [N][d] for visual steps 0..N-1 and kc, vc [C][d]."""
    t, bb, hh = _grid(0, wl.num_visual, [b], [h], "cpu")
    q, k, v = _visual(wl, layer, t, bb, hh, seed, "cpu")
    tc, bb, hh = _grid(0, wl.prefix_len, [b], [h], "cpu")
    tc = tc + wl.num_visual
    kc = _noise(wl, T_KC, layer, tc, bb, hh, seed, "cpu").to(torch.bfloat16)
    vc = _noise(wl, T_VC, layer, tc, bb, hh, seed, "cpu").to(torch.bfloat16)
    return (q[:, 0, 0], k[:, 0, 0], v[:, 0, 0], kc[:, 0, 0], vc[:, 0, 0])

"""ctypes binding of libheadkv.so: the C ABI of include/headkv.h, one Python
function per entry point under the same name.  Argument marshalling only --
every step of the decode path runs in the library's HIP kernels; if the
library is not built, loading fails loudly instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence, Tuple

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libheadkv.so")

HEADKV_OK = 0
HEADKV_ERR_INVALID_ARG = -1
HEADKV_ERR_CAPACITY = -2
HEADKV_ERR_STATE = -3
HEADKV_ERR_HIP = -4
HEADKV_ERR_UNSUPPORTED = -5

HEADKV_BUDGET_PAPER = 0
HEADKV_BUDGET_OVERRIDE = 1
HEADKV_BUDGET_TOTAL = 2

HEADKV_SCORE_MEAN_LOGIT = 0
HEADKV_SCORE_ATTN_SUM = 1

HEADKV_MAX_VISUAL = 16384
HEADKV_MAX_PREFIX = 2048
HEADKV_MAX_CAPACITY = 4608

HEADKV_TIMED_ATTN_APPEND = 0        # fused append + attention, compressed cache
HEADKV_TIMED_ATTN = 1               # attention after an update
HEADKV_TIMED_UPDATE = 2             # append + periodic update
HEADKV_TIMED_PREFILL = 3            # prefix store + causal prefix attention
HEADKV_TIMED_ATTN_APPEND_DENSE = 4  # fused append + attention before grouping
HEADKV_TIMED_UPDATE_ATTN = 5        # append + periodic update + attention, one launch
HEADKV_TIMED_KINDS = 6

HEADKV_ATTN_VARLEN = 0
HEADKV_ATTN_PADDED = 1
HEADKV_ATTN_GROUPED = 2
ATTN_STRATEGIES = {"varlen": HEADKV_ATTN_VARLEN, "padded": HEADKV_ATTN_PADDED,
                   "grouped": HEADKV_ATTN_GROUPED}

EXPORTED = (
    "headkv_plan", "headkv_create", "headkv_destroy", "headkv_prefill", "headkv_prefill_attn",
    "headkv_append_and_evict", "headkv_score_heads", "headkv_assign_budgets",
    "headkv_decode_attn", "headkv_decode_attn_noalloc", "headkv_decode_attn_layers",
    "headkv_decode_step",
    "headkv_export_retained",
    "headkv_run_steps", "headkv_timing_reserve", "headkv_timing_collect",
    "headkv_last_error",
)


class HeadKVConfig(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("num_layers", ctypes.c_int32),
        ("num_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("prefix_len", ctypes.c_int32), ("row_len", ctypes.c_int32),
        ("num_visual", ctypes.c_int32), ("recent_len", ctypes.c_int32),
        ("local_window", ctypes.c_int32), ("period", ctypes.c_int32),
        ("group_threshold", ctypes.c_int32), ("budget_mode", ctypes.c_int32),
        ("rho_num", ctypes.c_int32), ("rho_den", ctypes.c_int32),
        ("rs_num", ctypes.c_int32), ("rs_den", ctypes.c_int32),
        ("attn_strategy", ctypes.c_int32), ("score_mode", ctypes.c_int32),
        ("cfg_pairs", ctypes.c_int32),
        ("tau", ctypes.c_double),
    ]


class HeadKVError(RuntimeError):
    def __init__(self, status: int, what: str, msg: str):
        super().__init__(f"{what} failed with status {status}: {msg}")
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run paper_2605_20600_amd.build.build() "
                           "(or __graft_entry__.build()) first")
    L = ctypes.CDLL(LIB_PATH)
    P, I, Z = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    cfgp = ctypes.POINTER(HeadKVConfig)
    sig = {
        "headkv_plan": [cfgp, ctypes.POINTER(Z), ctypes.POINTER(Z), ctypes.POINTER(Z)],
        "headkv_create": [cfgp, P, P, P, ctypes.POINTER(P)],
        "headkv_prefill": [P, I, P, P, P],
        "headkv_prefill_attn": [P, I, P, P, P, P, P],
        "headkv_append_and_evict": [P, I, I, P, P, P, P],
        "headkv_score_heads": [P, I, P, P, P, P],
        "headkv_assign_budgets": [P, I, P, P, P, P, Z, ctypes.POINTER(Z), P],
        "headkv_decode_attn": [P, I, P, P, P],
        "headkv_decode_attn_noalloc": [P, I, P, P, P],
        "headkv_decode_step": [P, I, I, P, P, P, P, P],
        "headkv_decode_attn_layers": [P, I, I, P, P, P],
        "headkv_export_retained": [P, I, P, P, P],
        "headkv_run_steps": [P, I, I, P, P, P, ctypes.c_int64, P, I, P],
        "headkv_timing_reserve": [P, ctypes.c_int64],
        "headkv_timing_collect": [P, P, P, P, ctypes.POINTER(ctypes.c_int64)],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = ctypes.c_int32
    L.headkv_destroy.argtypes = [P]
    L.headkv_destroy.restype = None
    L.headkv_last_error.argtypes = []
    L.headkv_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def headkv_last_error() -> str:
    return load().headkv_last_error().decode()


def _check(status: int, what: str) -> int:
    if status != HEADKV_OK:
        raise HeadKVError(status, what, headkv_last_error())
    return status


def headkv_plan(cfg: HeadKVConfig) -> Tuple[int, int, int]:
    d, m, w = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check(load().headkv_plan(ctypes.byref(cfg), ctypes.byref(d), ctypes.byref(m), ctypes.byref(w)),
           "headkv_plan")
    return d.value, m.value, w.value


def headkv_create(cfg: HeadKVConfig, dense_kv: Sequence[int], meta: Sequence[int],
                  workspace: int) -> int:
    n = len(dense_kv)
    dk = (ctypes.c_void_p * n)(*dense_kv)
    me = (ctypes.c_void_p * n)(*meta)
    out = ctypes.c_void_p()
    _check(load().headkv_create(ctypes.byref(cfg), dk, me, workspace, ctypes.byref(out)),
           "headkv_create")
    return out.value


def headkv_destroy(h: int) -> None:
    load().headkv_destroy(h)


def headkv_prefill(h: int, layer: int, k_c: int, v_c: int, stream: int = 0) -> None:
    _check(load().headkv_prefill(h, layer, k_c, v_c, stream), "headkv_prefill")


def headkv_prefill_attn(h: int, layer: int, q_c: int, k_c: int, v_c: int, out_c: int,
                        stream: int = 0) -> None:
    _check(load().headkv_prefill_attn(h, layer, q_c, k_c, v_c, out_c, stream), "headkv_prefill_attn")


def headkv_append_and_evict(h: int, layer: int, step: int, q: int, k: int, v: int,
                            stream: int = 0) -> None:
    _check(load().headkv_append_and_evict(h, layer, step, q, k, v, stream),
           "headkv_append_and_evict")


def headkv_score_heads(h: int, layer: int, q: int, n_star: int, is_local: int,
                       stream: int = 0) -> None:
    _check(load().headkv_score_heads(h, layer, q, n_star, is_local, stream), "headkv_score_heads")


def headkv_assign_budgets(h: int, layer: int, is_local: int, budget_override: Optional[int],
                          budgets: int, ragged_kv: Optional[int], ragged_bytes: int,
                          stream: int = 0) -> Tuple[int, int]:
    """Returns (status, ragged_bytes_needed); HEADKV_ERR_CAPACITY is returned,
    not raised, so the caller can allocate and call again."""
    need = ctypes.c_size_t()
    st = load().headkv_assign_budgets(h, layer, is_local, budget_override, budgets, ragged_kv,
                                      ragged_bytes, ctypes.byref(need), stream)
    if st not in (HEADKV_OK, HEADKV_ERR_CAPACITY):
        _check(st, "headkv_assign_budgets")
    return st, need.value


def headkv_decode_attn(h: int, layer: int, q: int, out: int, stream: int = 0) -> None:
    _check(load().headkv_decode_attn(h, layer, q, out, stream), "headkv_decode_attn")


def headkv_decode_attn_noalloc(h: int, layer: int, q: int, out: int, stream: int = 0) -> None:
    _check(load().headkv_decode_attn_noalloc(h, layer, q, out, stream),
           "headkv_decode_attn_noalloc")


def headkv_decode_attn_layers(h: int, layer_begin: int, layer_end: int, q: Sequence[int],
                              out: Sequence[int], stream: int = 0) -> None:
    n = layer_end - layer_begin
    qa = (ctypes.c_void_p * n)(*q)
    oa = (ctypes.c_void_p * n)(*out)
    _check(load().headkv_decode_attn_layers(h, layer_begin, layer_end, qa, oa, stream),
           "headkv_decode_attn_layers")


def headkv_decode_step(h: int, layer: int, step: int, q: int, k: int, v: int, out: int,
                       stream: int = 0) -> None:
    _check(load().headkv_decode_step(h, layer, step, q, k, v, out, stream), "headkv_decode_step")


def headkv_export_retained(h: int, layer: int, mask: int, count: int, stream: int = 0) -> None:
    _check(load().headkv_export_retained(h, layer, mask, count, stream), "headkv_export_retained")


def headkv_run_steps(h: int, step_begin: int, step_end: int, q: Sequence[int], k: Sequence[int],
                     v: Sequence[int], step_stride: int, out: Sequence[int],
                     timing_every: int = 0, stream: int = 0) -> None:
    n = len(q)
    arr = lambda xs: (ctypes.c_void_p * n)(*xs)
    _check(load().headkv_run_steps(h, step_begin, step_end, arr(q), arr(k), arr(v), step_stride,
                                   arr(out), timing_every, stream), "headkv_run_steps")


def headkv_timing_reserve(h: int, launches: int) -> None:
    _check(load().headkv_timing_reserve(h, launches), "headkv_timing_reserve")


def headkv_timing_collect(h: int):
    """Returns per kind (fused append + attention after grouping, attention
    after an update, append + update, prefill, fused append + attention before
    grouping, append + update + attention in one launch) a list of (kernel ms,
    launches, algorithmic bytes), and the dropped count."""
    K = HEADKV_TIMED_KINDS
    ms = (ctypes.c_double * K)()
    n = (ctypes.c_int64 * K)()
    b = (ctypes.c_double * K)()
    dr = ctypes.c_int64()
    _check(load().headkv_timing_collect(h, ms, n, b, ctypes.byref(dr)), "headkv_timing_collect")
    return [(ms[i], n[i], b[i]) for i in range(K)], dr.value

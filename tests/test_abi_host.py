"""Host-side checks of the C ABI: the library loads, exports every function the
header declares, and rejects bad arguments and out-of-order calls with the
documented status before touching the GPU.  No kernel is launched here."""
import ctypes
import os
import re

import pytest

from paper_2605_20600_amd import binding as B
from paper_2605_20600_amd import workloads as W
from paper_2605_20600_amd.session import make_config

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "headkv.h")
FAKE = 0x7F0000000000          # 256-byte aligned, never dereferenced by these calls


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(headkv_[a-z_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    lib = B.load()
    names = _declared()
    assert set(names) == set(B.EXPORTED), names
    for n in names:
        assert hasattr(lib, n), n


def _status(fn, *args):
    return getattr(B.load(), fn)(*args)


def test_plan_sizes_and_validation():
    cfg = make_config(W.LUMINA768)
    dense, meta, ws = B.headkv_plan(cfg)
    assert dense > 0 and meta > 0 and ws > 0
    # dense cache holds prefix + threshold tokens (K and V) for every head
    per_head = 2 * (128 + 300) * 128 * 2 + 300 * 4
    assert dense >= 8 * 32 * per_head
    bad = [dict(head_dim=96), dict(batch=0), dict(num_visual=0), dict(group_threshold=0),
           dict(group_threshold=99999), dict(period=0), dict(tau=0.0), dict(tau=1.5),
           dict(rho_num=0), dict(rho_num=3, rho_den=2), dict(rs_num=3, rs_den=2),
           dict(budget_mode=7), dict(prefix_len=-1), dict(row_len=0), dict(recent_len=0),
           dict(num_heads=2000), dict(attn_strategy=3), dict(attn_strategy=-1)]
    for kw in bad:
        c = make_config(W.LUMINA768)
        for k, v in kw.items():
            setattr(c, k, v)
        with pytest.raises(B.HeadKVError) as e:
            B.headkv_plan(c)
        assert e.value.status in (B.HEADKV_ERR_INVALID_ARG, B.HEADKV_ERR_UNSUPPORTED), kw
        assert B.headkv_last_error() != ""


def test_config_struct_matches_header():
    # the binding's struct mirrors headkv_config field by field
    src = open(HEADER).read()
    body = src[src.index("typedef struct headkv_config {"):src.index("} headkv_config;")]
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = []
    for decl in re.findall(r"(int32_t|double)\s+([^;]+);", body):
        fields += [(decl[0], n.strip()) for n in decl[1].split(",")]
    ct = {"int32_t": ctypes.c_int32, "double": ctypes.c_double}
    assert [(n, ct[t]) for t, n in fields] == list(B.HeadKVConfig._fields_)


def test_constants_match_header():
    # every integer constant the header defines has the same value in the binding
    src = open(HEADER).read()
    found = re.findall(r"#define (HEADKV_[A-Z_0-9]+) \(?(-?\d+)\)?", src)
    assert len(found) >= 20
    for name, value in found:
        assert getattr(B, name, None) == int(value), name


def _handle(wl=W.TINY):
    cfg = make_config(wl)
    return B.headkv_create(cfg, [FAKE] * cfg.num_layers, [FAKE + 4096] * cfg.num_layers, FAKE), cfg


def test_create_rejects_bad_buffers():
    cfg = make_config(W.TINY)
    with pytest.raises(B.HeadKVError) as e:
        B.headkv_create(cfg, [0], [FAKE], FAKE)
    assert e.value.status == B.HEADKV_ERR_INVALID_ARG
    with pytest.raises(B.HeadKVError) as e:
        B.headkv_create(cfg, [FAKE + 8], [FAKE], FAKE)
    assert e.value.status == B.HEADKV_ERR_INVALID_ARG
    with pytest.raises(B.HeadKVError):
        B.headkv_create(cfg, [FAKE], [FAKE], FAKE + 4)


def test_calls_out_of_order_are_state_errors():
    h, cfg = _handle()
    try:
        S = B.HEADKV_ERR_STATE
        assert _status("headkv_decode_attn", h, 0, FAKE, FAKE, None) == S
        assert _status("headkv_append_and_evict", h, 0, 0, FAKE, FAKE, FAKE, None) == S
        assert _status("headkv_score_heads", h, 0, FAKE, FAKE, FAKE, None) == S
        need = ctypes.c_size_t()
        assert _status("headkv_assign_budgets", h, 0, FAKE, None, FAKE, None, 0,
                       ctypes.byref(need), None) == S
        assert _status("headkv_export_retained", h, 0, FAKE, FAKE, None) == S
    finally:
        B.headkv_destroy(h)


def test_bad_arguments_are_rejected():
    h, cfg = _handle()
    try:
        I = B.HEADKV_ERR_INVALID_ARG
        assert _status("headkv_decode_attn", h, 5, FAKE, FAKE, None) == I      # layer
        assert _status("headkv_decode_attn", h, -1, FAKE, FAKE, None) == I
        assert _status("headkv_decode_attn", h, 0, None, FAKE, None) == I
        assert _status("headkv_prefill", h, 0, None, None, None) == I          # C = 32 > 0
        assert _status("headkv_prefill", h, 0, FAKE + 2, FAKE, None) == I      # misaligned
        assert _status("headkv_decode_attn", None, 0, FAKE, FAKE, None) == I   # handle
        assert _status("headkv_append_and_evict", h, 0, 0, None, FAKE, FAKE, None) == I
        need = ctypes.c_size_t()
        assert _status("headkv_assign_budgets", h, 0, None, None, FAKE, None, 0,
                       ctypes.byref(need), None) == I
    finally:
        B.headkv_destroy(h)


def test_misaligned_vectors_are_rejected():
    # the kernels read q, k, v rows and write outputs with 16-byte vector
    # accesses: every per-step vector must be 16-byte aligned
    h, cfg = _handle()
    try:
        I = B.HEADKV_ERR_INVALID_ARG
        assert _status("headkv_append_and_evict", h, 0, 0, FAKE + 2, FAKE, FAKE, None) == I
        assert _status("headkv_append_and_evict", h, 0, 0, FAKE, FAKE + 8, FAKE, None) == I
        assert _status("headkv_append_and_evict", h, 0, 0, FAKE, FAKE, FAKE + 4, None) == I
        assert _status("headkv_decode_step", h, 0, 0, FAKE, FAKE, FAKE, FAKE + 4, None) == I
        assert _status("headkv_decode_step", h, 0, 0, FAKE + 2, FAKE, FAKE, FAKE, None) == I
        assert _status("headkv_decode_attn", h, 0, FAKE + 2, FAKE, None) == I
        assert _status("headkv_decode_attn", h, 0, FAKE, FAKE + 4, None) == I
        assert _status("headkv_score_heads", h, 0, FAKE + 2, FAKE, FAKE, None) == I
        arr = (ctypes.c_void_p * 1)(FAKE)
        # a step stride of 3 elements would misalign every other step's rows
        assert _status("headkv_run_steps", h, 0, 1, arr, arr, arr, 3, arr, 0, None) == I
        bad = (ctypes.c_void_p * 1)(FAKE + 2)
        assert _status("headkv_run_steps", h, 0, 1, bad, arr, arr, 256, arr, 0, None) == I
        # aligned arguments get past the checks to the call-order error
        assert _status("headkv_decode_attn", h, 0, FAKE, FAKE, None) == B.HEADKV_ERR_STATE
    finally:
        B.headkv_destroy(h)
    wl = W.LUMINA768.with_(layers=2)
    h = B.headkv_create(make_config(wl), [FAKE] * 2, [FAKE + 4096] * 2, FAKE)
    try:
        ok = (ctypes.c_void_p * 2)(FAKE, FAKE)
        bad = (ctypes.c_void_p * 2)(FAKE, FAKE + 4)
        assert _status("headkv_decode_attn_layers", h, 0, 2, ok, bad, None) == \
            B.HEADKV_ERR_INVALID_ARG
    finally:
        B.headkv_destroy(h)


def test_override_mode_requires_budgets():
    wl = W.TINY.with_(budget_mode=W.BUDGET_OVERRIDE)
    h, cfg = _handle(wl)
    try:
        need = ctypes.c_size_t()
        assert _status("headkv_assign_budgets", h, 0, FAKE, None, FAKE, None, 0,
                       ctypes.byref(need), None) == B.HEADKV_ERR_INVALID_ARG
    finally:
        B.headkv_destroy(h)


def test_prefill_attention_and_multi_layer_arguments():
    h, cfg = _handle()
    try:
        I, U, S = B.HEADKV_ERR_INVALID_ARG, B.HEADKV_ERR_UNSUPPORTED, B.HEADKV_ERR_STATE
        assert _status("headkv_prefill_attn", h, 0, None, FAKE, FAKE, FAKE, None) == I
        assert _status("headkv_prefill_attn", h, 0, FAKE, FAKE, FAKE, None, None) == I
        assert _status("headkv_prefill_attn", h, 0, FAKE + 2, FAKE, FAKE, FAKE, None) == I
        arr = (ctypes.c_void_p * 1)(FAKE)
        assert _status("headkv_decode_attn_layers", h, 0, 2, arr, arr, None) == I   # range
        assert _status("headkv_decode_attn_layers", h, 0, 1, None, arr, None) == I
        # Tiny has 4 heads: fewer than the CUs the one-launch plan needs
        assert _status("headkv_decode_attn_layers", h, 0, 1, arr, arr, None) == U
    finally:
        B.headkv_destroy(h)
    wl = W.LUMINA768.with_(layers=2)
    cfg = make_config(wl)
    h = B.headkv_create(cfg, [FAKE] * 2, [FAKE + 4096] * 2, FAKE)
    try:
        arr = (ctypes.c_void_p * 2)(FAKE, FAKE)
        assert _status("headkv_decode_attn_layers", h, 0, 2, arr, arr, None) == B.HEADKV_ERR_STATE
    finally:
        B.headkv_destroy(h)


def test_cfg_pairs_need_an_even_batch():
    cfg = make_config(W.TINY)
    cfg.cfg_pairs = 1
    with pytest.raises(B.HeadKVError) as e:
        B.headkv_plan(cfg)
    assert e.value.status == B.HEADKV_ERR_INVALID_ARG
    cfg.batch = 2
    B.headkv_plan(cfg)

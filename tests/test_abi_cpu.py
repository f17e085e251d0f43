"""Host-side checks of the C ABI: the library loads, exports every declared
entry point, and rejects bad arguments before any GPU work is enqueued."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2606_14782_amd import bacon

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "bacon.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(bacon_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary_calls():
    names = _declared()
    for required in ("bacon_score", "bacon_calibrate", "bacon_select_topk", "bacon_compact",
                     "bacon_compress_layer"):
        assert required in names


def test_library_exports_every_declared_symbol():
    L = bacon.lib()
    missing = [n for n in _declared() if not hasattr(L, n)]
    assert not missing, f"not exported: {missing}"
    assert sorted(bacon.ENTRY_POINTS) == _declared()


def _shape(**kw):
    d = dict(num_layers=4, num_q_heads=8, num_kv_heads=2, head_dim=128, window=32, max_batch=2,
             max_total_tokens=4096, dtype=bacon.BF16)
    d.update(kw)
    return bacon.Shape(**d)


def _ws(shape, params=None):
    p = params or bacon.default_params()
    return bacon.lib().bacon_workspace_bytes(C.byref(shape), C.byref(p))


def test_defaults_follow_the_paper():
    p = bacon.default_params()
    assert (p.radius, p.persist_m, p.rho) == (5, 4, 2.0)
    assert p.gamma == 1.0 and p.use_last_query == 1 and p.terms == 7
    assert p.pool_kernel % 2 == 1
    assert p.pool_mode == bacon.POOL_MEAN_S
    assert p.head_alloc == bacon.ALLOC_GIVEN and abs(p.alloc_floor - 0.2) < 1e-7


@pytest.mark.parametrize("kw,expect_zero", [
    ({}, False),
    ({"num_q_heads": 7}, True),            # not a multiple of num_kv_heads
    ({"head_dim": 96}, True),              # unsupported head dim
    ({"window": 0}, True),
    ({"max_batch": 65}, True),
    ({"dtype": 7}, True),
    ({"num_q_heads": 32, "num_kv_heads": 2, "window": 32}, True),   # G*W = 512 > 256
])
def test_workspace_size_validates_shape(kw, expect_zero):
    n = _ws(_shape(**kw))
    assert (n == 0) == expect_zero
    if expect_zero:
        assert bacon.lib().bacon_last_error()


@pytest.mark.parametrize("kw", [{"radius": -1}, {"radius": 17}, {"persist_m": 17}, {"rho": 0.0},
                                {"gamma": -1.0}, {"pool_kernel": 4}, {"pool_kernel": 35},
                                {"use_last_query": 2}, {"terms": 8}, {"pool_mode": -1},
                                {"pool_mode": 3}, {"head_alloc": 2}, {"alloc_floor": -0.1},
                                {"alloc_floor": 1.5}])
def test_bad_params_rejected(kw):
    assert _ws(_shape(), bacon.default_params(**kw)) == 0


def test_workspace_grows_with_tokens_and_depth():
    a = _ws(_shape())
    b = _ws(_shape(max_total_tokens=8192))
    c = _ws(_shape(), bacon.default_params(persist_m=8))
    assert 0 < a < b and a < c


def _init(shape=None, ws_bytes=None, align=256):
    shape = shape or _shape()
    n = _ws(shape)
    h = C.c_void_p()
    fake = C.c_void_p(0x100000 + (align if align != 256 else 0))
    st = bacon.lib().bacon_init(C.byref(h), C.byref(shape), None, fake,
                                n if ws_bytes is None else ws_bytes)
    return st, h


def test_init_checks_workspace_without_touching_the_gpu():
    st, _ = _init(ws_bytes=16)
    assert st == bacon.ERR_WORKSPACE
    st, _ = _init(align=16)
    assert st == bacon.ERR_WORKSPACE
    st, h = _init()
    assert st == bacon.OK and h.value
    bacon.lib().bacon_free(h)


def _batch(cu, budgets):
    return bacon.BatchLayout(cu, budgets)


def test_calls_reject_bad_batches_and_order_before_enqueueing():
    st, h = _init()
    assert st == bacon.OK
    L = bacon.lib()
    fake = C.c_void_p(0x200000)
    good = _batch([0, 1000, 3000], [64, 128])
    # no prompt begun -> ORDER
    assert L.bacon_compress_layer(h, 0, C.byref(good.c), fake, fake, fake, fake, fake, fake,
                                  None) == bacon.ERR_ORDER
    assert L.bacon_compress_layer_lse(h, 0, C.byref(good.c), fake, fake, fake, fake, fake, fake,
                                      fake, None) == bacon.ERR_ORDER
    # NULL or misaligned normalisers
    assert L.bacon_compress_layer_lse(h, 0, C.byref(good.c), fake, fake, fake, None, fake, fake,
                                      fake, None) == bacon.ERR_INVALID
    assert L.bacon_compress_layer_lse(h, 0, C.byref(good.c), fake, fake, fake,
                                      C.c_void_p(0x200002), fake, fake, fake,
                                      None) == bacon.ERR_INVALID
    # sequence shorter than the window
    assert L.bacon_score(h, 0, C.byref(_batch([0, 10], [4]).c), fake, fake, None, fake, fake,
                         None) == bacon.ERR_INVALID
    # prompt call: pointer arrays, layer range, order
    arr1 = (C.c_void_p * 1)(0x200000)
    assert L.bacon_compress_prompt(h, C.byref(good.c), 0, 1, None, arr1, arr1, None, arr1, arr1,
                                   arr1, None, None) == bacon.ERR_INVALID
    assert L.bacon_compress_prompt(h, C.byref(good.c), 0, 0, arr1, arr1, arr1, None, arr1, arr1,
                                   arr1, None, None) == bacon.ERR_INVALID
    assert L.bacon_compress_prompt(h, C.byref(good.c), 1, 1, arr1, arr1, arr1, None, arr1, arr1,
                                   arr1, None, None) == bacon.ERR_ORDER
    assert L.bacon_compress_prompt(h, C.byref(good.c), 0, 9, arr1, arr1, arr1, None, arr1, arr1,
                                   arr1, None, None) == bacon.ERR_ORDER
    bad = (C.c_void_p * 1)(0x200002)
    assert L.bacon_compress_prompt(h, C.byref(good.c), 0, 1, arr1, arr1, arr1, bad, arr1, arr1,
                                   arr1, None, None) == bacon.ERR_INVALID
    # no prompt begun -> ORDER, before anything is enqueued
    assert L.bacon_compress_prompt(h, C.byref(good.c), 0, 1, arr1, arr1, arr1, None, arr1, arr1,
                                   arr1, None, None) == bacon.ERR_ORDER
    # a per-layer batch array with a NULL entry
    nolb = (C.c_void_p * 1)(None)
    assert L.bacon_compress_prompt(h, C.byref(good.c), 0, 1, arr1, arr1, arr1, None, arr1, arr1,
                                   arr1, nolb, None) == bacon.ERR_INVALID
    # capture buffers: all three or none
    assert L.bacon_debug_capture(h, fake, None, fake) == bacon.ERR_INVALID
    assert L.bacon_debug_capture(h, fake, fake, C.c_void_p(0x200002)) == bacon.ERR_INVALID
    assert L.bacon_debug_capture(h, None, None, None) == bacon.OK
    # the static-scratch normalisers: a batch whose scratch exceeds the static
    # array is refused before the GPU is touched; a bad shape is refused
    wide = _shape(num_q_heads=256, num_kv_heads=64, window=32, max_total_tokens=1 << 20,
                  max_batch=1)
    assert L.bacon_window_lse_static(C.byref(wide), C.byref(_batch([0, 32768], [4]).c), fake, fake,
                                     fake, None) == bacon.ERR_WORKSPACE
    assert b"static scratch" in L.bacon_last_error()
    assert L.bacon_window_lse_static(C.byref(_shape(head_dim=96)), C.byref(good.c), fake, fake, fake,
                                     None) == bacon.ERR_UNSUPPORTED
    assert L.bacon_window_lse_static(None, C.byref(good.c), fake, fake, fake,
                                     None) == bacon.ERR_INVALID
    # window normalisers alone: NULL or misaligned pointers, short sequences
    assert L.bacon_window_lse(h, C.byref(good.c), fake, fake, None, None) == bacon.ERR_INVALID
    assert L.bacon_window_lse(h, C.byref(good.c), fake, fake, C.c_void_p(0x200002),
                              None) == bacon.ERR_INVALID
    assert L.bacon_window_lse(h, C.byref(good.c), None, fake, fake, None) == bacon.ERR_INVALID
    assert L.bacon_window_lse(h, C.byref(_batch([0, 10], [4]).c), fake, fake, fake,
                              None) == bacon.ERR_INVALID
    assert L.bacon_window_lse(None, C.byref(good.c), fake, fake, fake, None) == bacon.ERR_INVALID
    # too many tokens for the context
    assert L.bacon_score(h, 0, C.byref(_batch([0, 5000], [4]).c), fake, fake, None, fake, fake,
                         None) == bacon.ERR_INVALID
    # budget < 1
    assert L.bacon_select_topk(h, C.byref(_batch([0, 100], [0]).c), fake, fake,
                               None) == bacon.ERR_INVALID
    # cu_seqlens[0] != 0
    assert L.bacon_select_topk(h, C.byref(_batch([5, 100], [4]).c), fake, fake,
                               None) == bacon.ERR_INVALID
    # NULL and misaligned pointers
    assert L.bacon_score(h, 0, C.byref(good.c), None, fake, None, fake, fake,
                         None) == bacon.ERR_INVALID
    assert L.bacon_compact(h, C.byref(good.c), C.c_void_p(0x200004), fake, fake, fake, fake,
                           None) == bacon.ERR_INVALID
    # layer out of range
    assert L.bacon_score(h, 9, C.byref(good.c), fake, fake, None, fake, fake,
                         None) == bacon.ERR_INVALID
    assert b"layer" in L.bacon_last_error()
    # adaptive allocation: NULL or misaligned pointers, head budgets given,
    # and the output switch
    assert L.bacon_allocate_heads(h, C.byref(good.c), None, fake, None) == bacon.ERR_INVALID
    assert L.bacon_allocate_heads(h, C.byref(good.c), fake, C.c_void_p(0x200002),
                                  None) == bacon.ERR_INVALID
    hb = bacon.BatchLayout([0, 1000, 3000], [64, 128], head_budgets=np.full((2, 2), 8))
    assert L.bacon_allocate_heads(h, C.byref(hb.c), fake, fake, None) == bacon.ERR_INVALID
    assert b"per-sequence" in L.bacon_last_error()
    assert L.bacon_allocate_heads(None, C.byref(good.c), fake, fake, None) == bacon.ERR_INVALID
    assert L.bacon_alloc_output(h, C.c_void_p(0x200002)) == bacon.ERR_INVALID
    assert L.bacon_alloc_output(h, fake) == bacon.OK
    assert L.bacon_alloc_output(h, None) == bacon.OK
    # too long a sequence for the select kernel
    big = _init(_shape(max_total_tokens=70000, max_batch=1))[1]
    assert L.bacon_select_topk(big, C.byref(_batch([0, 40000], [4]).c), fake, fake,
                               None) == bacon.ERR_UNSUPPORTED
    L.bacon_free(big)
    L.bacon_free(h)


def test_output_sizes():
    b = _batch([0, 1000, 3000, 3500], [64, 128, 512])
    assert b.idx_count(8) == (64 + 128 + 512) * 8
    assert b.kept_rows(32) == 64 + 128 + 512 + 3 * 32


def test_status_strings():
    L = bacon.lib()
    for s in range(6):
        assert L.bacon_status_string(s)


def test_counts_with_head_budgets():
    """idx entries and compacted rows with a budget per (sequence, KV head)."""
    hb = np.array([[3, 7], [5, 1]], np.int32)
    b = bacon.BatchLayout([0, 100, 300], [4, 4], head_budgets=hb)
    assert b.idx_count(2) == 3 + 7 + 5 + 1
    assert b.kept_rows(8, 2) == (7 + 8) + (5 + 8)
    u = bacon.BatchLayout([0, 100, 300], [4, 6])
    assert u.idx_count(2) == 2 * (4 + 6) and u.kept_rows(8, 2) == (4 + 8) + (6 + 8)

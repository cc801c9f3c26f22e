"""Calls of the C ABI that pass validation, for the sanitizer build only
(its launches are stand-ins that check the host layer's launch arguments;
with the real library these calls would launch kernels). Run by
tests/test_sanitize_cpu.py in a process with AddressSanitizer preloaded."""
import ctypes

import pytest

from paper_2607_03612_amd import binding as B

OK = ctypes.c_void_p(0x10000)  # never dereferenced by the stand-ins


def _p(heads, frames, T, dtype=B.BF16):
    return B.Problem(heads, frames, T, 64, 64, dtype)


TABLES = [
    # every class on a small ragged layer
    (12, 3, 261, [(B.DENSE, 0), (B.FRAME_LOCAL, 0), (B.TOPK, 5), (B.ANCHOR, 0), (B.ANCHOR, 2),
                  (B.STRIDE, 1), (B.STRIDE, 7), (B.STRIDE, 783), (B.GLOBAL_PROBE, 3),
                  (B.COSINE_TOPK, 1), (B.COSINE_TOPK, 2), (B.SKIP, 0)]),
    # the split: a 274800-token layer with long lists and a dense head
    (6, 200, 1374, [(B.TOPK, 959), (B.GLOBAL_PROBE, 400), (B.COSINE_TOPK, 3), (B.DENSE, 0),
                    (B.FRAME_LOCAL, 0), (B.STRIDE, 9)]),
    # the largest problem: 2^20 tokens, the most blocks
    (3, 8, 131072, [(B.TOPK, 164), (B.FRAME_LOCAL, 0), (B.TOPK, 16384)]),
    # the most heads, cycling through the classes
    (256, 2, 300, [[(B.DENSE, 0), (B.FRAME_LOCAL, 0), (B.TOPK, 3), (B.ANCHOR, 1), (B.STRIDE, 5),
                    (B.GLOBAL_PROBE, 2), (B.COSINE_TOPK, 1), (B.SKIP, 0)][h % 8] for h in range(256)]),
]


@pytest.mark.parametrize("heads,frames,T,table", TABLES)
@pytest.mark.parametrize("dtype", [B.BF16, B.F32])
def test_valid_calls_reach_consistent_launches(heads, frames, T, table, dtype):
    lib = B.load()
    p = _p(heads, frames, T, dtype)
    t = B.head_table(table)
    cap = lib.saf3r_index_capacity(ctypes.byref(p), t)
    assert cap >= 1
    assert lib.saf3r_estimate_blocks(ctypes.byref(p), t, OK, OK, OK, OK, None) == 0
    sel = lib.saf3r_select_blocks
    ws = lib.saf3r_select_workspace_bytes(ctypes.byref(p), t)
    # single-launch path (when its score rows fit in LDS), full and one-head workspaces
    nb = lib.saf3r_num_blocks(ctypes.byref(p))
    if nb <= 8192:
        assert sel(ctypes.byref(p), t, OK, OK, OK, OK, cap, None, None, 0, None) == 0
    assert sel(ctypes.byref(p), t, OK, OK, OK, OK, cap, OK, OK, max(ws, 16), None) == 0
    n_topk = sum(1 for c, _ in table if c == B.TOPK)
    if n_topk > 1:
        assert sel(ctypes.byref(p), t, OK, OK, OK, OK, cap, None, OK, ws // n_topk, None) == 0
    att = lib.saf3r_sparse_attention
    aws = lib.saf3r_attention_workspace_bytes(ctypes.byref(p), t)
    assert att(ctypes.byref(p), t, OK, OK, OK, OK, OK, cap, OK, OK, None, 0, None) == 0
    assert att(ctypes.byref(p), t, OK, OK, OK, OK, OK, cap, OK, None, OK, max(aws, 16), None) == 0
    if any(c == B.COSINE_TOPK for c, _ in table):
        cws = lib.saf3r_cosine_workspace_bytes(ctypes.byref(p), 96)
        assert lib.saf3r_cosine_select(ctypes.byref(p), t, OK, 96, OK, cws, OK, OK, cap, None) == 0
    nws = lib.saf3r_nmse_workspace_bytes(ctypes.byref(p))
    assert lib.saf3r_nmse(ctypes.byref(p), OK, OK, OK, nws, OK, None) == 0
    assert lib.saf3r_nmse_noalloc(ctypes.byref(p), OK, OK, OK, None) == 0


def test_all_dense_table_is_one_launch():
    lib = B.load()
    p = _p(16, 100, 1374)
    t = B.head_table([(B.DENSE, 0)] * 16)
    assert lib.saf3r_sparse_attention(ctypes.byref(p), t, OK, OK, OK, None, None, 0, OK, None,
                                      None, 0, None) == 0


@pytest.mark.parametrize("heads,frames,T,table", TABLES)
def test_list_check_reaches_a_consistent_launch(heads, frames, T, table):
    lib = B.load()
    p = _p(heads, frames, T)
    t = B.head_table(table)
    cap = lib.saf3r_index_capacity(ctypes.byref(p), t)
    first = ctypes.c_int32(-1)
    assert lib.saf3r_validate_index(ctypes.byref(p), t, OK, OK, cap, OK, ctypes.byref(first), None) == 0

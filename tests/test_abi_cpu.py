"""The C ABI on the host: the library loads, exports every declared symbol,
and rejects bad arguments with a status code before anything is launched
(none of these calls reaches the GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "saf3r.h")


@pytest.fixture(scope="module")
def B():
    from paper_2607_03612_amd import binding

    if not os.path.exists(binding.LIB_PATH):
        from paper_2607_03612_amd import build

        build.build()
    binding.load()
    return binding


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]*?\b(saf3r_\w+)\s*\(", text, re.M)))


def test_header_declares_the_three_hot_path_calls():
    names = declared_functions()
    for n in ("saf3r_estimate_blocks", "saf3r_select_blocks", "saf3r_sparse_attention"):
        assert n in names


def test_library_exports_every_declared_symbol(B):
    lib = ctypes.CDLL(B.LIB_PATH)
    names = declared_functions()
    assert set(names) == set(B.EXPORTS)
    for n in names:
        assert hasattr(lib, n), f"{n} is declared but not exported"


def _p(B, heads=16, frames=8, T=1374, head_dim=64, block=64, dtype=1):
    return B.Problem(heads, frames, T, head_dim, block, dtype)


def test_problem_validation(B):
    lib = B.load()
    nb = lib.saf3r_num_blocks
    assert nb(ctypes.byref(_p(B))) == 172
    assert nb(None) == -1
    assert nb(ctypes.byref(_p(B, heads=0))) == -1
    assert nb(ctypes.byref(_p(B, frames=-1))) == -1
    assert nb(ctypes.byref(_p(B, dtype=7))) == -1
    assert nb(ctypes.byref(_p(B, head_dim=128))) == -2
    assert nb(ctypes.byref(_p(B, block=128))) == -2
    assert nb(ctypes.byref(_p(B, heads=257))) == -2
    assert nb(ctypes.byref(_p(B, frames=1024, T=1025))) == -2  # > 2^20 tokens
    assert nb(ctypes.byref(_p(B, frames=1024, T=1024))) == 16384


def test_table_validation_and_capacity(B):
    lib = B.load()
    cap = lib.saf3r_index_capacity
    p = _p(B, heads=3, frames=8, T=1374)
    assert cap(ctypes.byref(p), B.head_table([(0, 0), (1, 0), (2, 13)])) == 44
    assert cap(ctypes.byref(p), B.head_table([(0, 0), (0, 0), (2, 100)])) == 100
    assert cap(ctypes.byref(p), B.head_table([(0, 0)] * 3)) == 1
    assert cap(ctypes.byref(p), B.head_table([(0, 0), (2, 0), (2, 1)])) == -5
    assert cap(ctypes.byref(p), B.head_table([(0, 0), (2, 173), (2, 1)])) == -5
    assert cap(ctypes.byref(p), B.head_table([(0, 0), (8, 1), (2, 1)])) == -5  # unknown class
    assert cap(ctypes.byref(p), B.head_table([(0, 0), (-1, 1), (2, 1)])) == -5
    assert cap(ctypes.byref(p), None) == -1
    # frames of 128 tokens align with blocks: two blocks per frame
    assert cap(ctypes.byref(_p(B, heads=1, frames=4, T=128)), B.head_table([(1, 0)])) == 2
    # one 300-token frame: every block shares it
    assert cap(ctypes.byref(_p(B, heads=1, frames=1, T=300)), B.head_table([(1, 0)])) == 5


def test_new_classes_validation_and_capacity(B):
    lib = B.load()
    cap = lib.saf3r_index_capacity
    p = _p(B, heads=2, frames=8, T=1374)  # N = 10992, nb = 172
    # ANCHOR: frame index in [0, frames); frame 0 = tokens 0..1373 -> blocks 0..21;
    # frame 3 = tokens 4122..5495 -> blocks 64..85
    assert cap(ctypes.byref(p), B.head_table([(B.ANCHOR, 0), (0, 0)])) == 22
    assert cap(ctypes.byref(p), B.head_table([(B.ANCHOR, 3), (0, 0)])) == 22
    assert cap(ctypes.byref(p), B.head_table([(B.ANCHOR, 7), (0, 0)])) == 22
    assert cap(ctypes.byref(p), B.head_table([(B.ANCHOR, 8), (0, 0)])) == -5
    assert cap(ctypes.byref(p), B.head_table([(B.ANCHOR, -1), (0, 0)])) == -5
    # STRIDE: key stride in [1, N]; no list
    assert cap(ctypes.byref(p), B.head_table([(B.STRIDE, 64), (0, 0)])) == 1
    assert cap(ctypes.byref(p), B.head_table([(B.STRIDE, 10992), (0, 0)])) == 1
    assert cap(ctypes.byref(p), B.head_table([(B.STRIDE, 0), (0, 0)])) == -5
    assert cap(ctypes.byref(p), B.head_table([(B.STRIDE, 10993), (0, 0)])) == -5
    # GLOBAL_PROBE: kept blocks in [1, nb]
    assert cap(ctypes.byref(p), B.head_table([(B.GLOBAL_PROBE, 40), (2, 7)])) == 40
    assert cap(ctypes.byref(p), B.head_table([(B.GLOBAL_PROBE, 172), (0, 0)])) == 172
    assert cap(ctypes.byref(p), B.head_table([(B.GLOBAL_PROBE, 173), (0, 0)])) == -5
    assert cap(ctypes.byref(p), B.head_table([(B.GLOBAL_PROBE, 0), (0, 0)])) == -5
    # a table of DENSE and STRIDE heads needs no lists: attention accepts null lists
    fake = ctypes.c_void_p(0x1000)
    t = B.head_table([(B.STRIDE, 4), (0, 0)])
    assert lib.saf3r_sparse_attention(ctypes.byref(p), t, fake, fake, fake, None, None, 0,
                                      None, None, None, 0, None) == -1  # out missing, lists not required


def test_calls_reject_bad_arguments_before_launch(B):
    lib = B.load()
    p = _p(B, heads=2, frames=2, T=100)
    t = B.head_table([(1, 0), (2, 2)])
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    assert lib.saf3r_estimate_blocks(ctypes.byref(p), t, None, fake, fake, fake, None) == -1
    assert lib.saf3r_estimate_blocks(ctypes.byref(_p(B, head_dim=32)), t, fake, fake, fake, fake, None) == -2
    sel = lib.saf3r_select_blocks
    assert sel(ctypes.byref(p), t, fake, fake, fake, fake, 3, None, None, 0, None) == -3
    assert sel(ctypes.byref(p), t, fake, None, fake, fake, 8, None, None, 0, None) == -1
    assert sel(ctypes.byref(p), B.head_table([(1, 0), (2, 9)]),
               fake, fake, fake, fake, 8, None, None, 0, None) == -5
    # workspace: one TOPK head of nb = 4 blocks takes 4 rows of 64 x 4 words
    need = lib.saf3r_select_workspace_bytes(ctypes.byref(p), t)
    assert need == 4 * 64 * 4 * 4
    assert lib.saf3r_select_workspace_bytes(ctypes.byref(p), B.head_table([(1, 0), (0, 0)])) == 0
    assert lib.saf3r_select_workspace_bytes(None, t) == -1
    assert sel(ctypes.byref(p), t, fake, fake, fake, fake, 8, None, fake, need - 16, None) == -3
    assert sel(ctypes.byref(p), t, fake, fake, fake, fake, 8, None, fake, -1, None) == -1
    assert lib.saf3r_sparse_attention(ctypes.byref(p), t, fake, fake, fake, fake, fake, 4,
                                      None, None, None, 0, None) == -1
    assert lib.saf3r_sparse_attention(ctypes.byref(p), t, fake, fake, fake, None, fake, 4,
                                      fake, None, None, 0, None) == -1
    assert lib.saf3r_sparse_attention(ctypes.byref(p), t, fake, fake, fake, fake, fake, 1,
                                      fake, None, None, 0, None) == -3


def test_attention_workspace_bytes_and_validation(B):
    """Split of long lists (Sec. 4.1 attention over kept blocks): on layers
    of 4096 or more key blocks, bf16 list heads that can keep 384 or more
    key blocks take 4 x nb items of 64 x 64 fp32 accumulators plus 64
    (max, sum) pairs each."""
    lib = B.load()
    size = lib.saf3r_attention_workspace_bytes
    item = 64 * 64 * 4 + 64 * 2 * 4
    p = _p(B, heads=4, frames=64, T=4096)  # nb = 4096, 64 blocks per frame
    t = B.head_table([(B.TOPK, 384), (B.TOPK, 383), (B.FRAME_LOCAL, 0), (B.DENSE, 0)])
    assert size(ctypes.byref(p), t) == 1 * 4 * 4096 * item
    both = B.head_table([(B.TOPK, 600), (B.GLOBAL_PROBE, 384), (B.COSINE_TOPK, 6), (B.STRIDE, 2)])
    assert size(ctypes.byref(p), both) == 3 * 4 * 4096 * item  # cosine: 6 x 64 frames = 384
    small = B.head_table([(B.COSINE_TOPK, 5), (B.ANCHOR, 0), (B.SKIP, 0), (B.DENSE, 0)])
    assert size(ctypes.byref(p), small) == 0
    assert size(ctypes.byref(_p(B, heads=4, frames=64, T=4096, dtype=B.F32)), t) == 0
    # a shorter layer (nb = 4095) splits nothing, whatever the lists
    assert size(ctypes.byref(_p(B, heads=4, frames=63, T=4160)), both) == 0
    assert size(None, t) == -1
    fake = ctypes.c_void_p(0x1000)
    need = 4 * 4096 * item
    att = lib.saf3r_sparse_attention
    assert att(ctypes.byref(p), t, fake, fake, fake, fake, fake, 384, fake, None,
               fake, need - 1, None) == -3
    assert att(ctypes.byref(p), t, fake, fake, fake, fake, fake, 384, fake, None,
               ctypes.c_void_p(0x1008), need, None) == -1
    nosplit = B.head_table([(B.TOPK, 100), (B.FRAME_LOCAL, 0), (B.DENSE, 0), (B.DENSE, 0)])
    assert att(ctypes.byref(p), nosplit, fake, fake, fake, fake, fake, 100, fake, None,
               fake, -1, None) == -1  # a negative size is rejected even when nothing splits
    assert att(ctypes.byref(p), t, fake, fake, fake, fake, fake, 383, fake, None,
               fake, need, None) == -3  # cap below the table's capacity fails first

def test_status_strings(B):
    lib = B.load()
    for s in (0, -1, -2, -3, -4, -5, -6, 42):
        assert lib.saf3r_status_string(s)
    assert lib.saf3r_status_string(-3).decode().startswith("index capacity or workspace")


def test_cosine_entry_points_validate_before_launch(B):
    lib = B.load()
    p = _p(B, heads=2, frames=8, T=1374)  # nb = 172
    # workspace: (feat_dim * nb + nb^2) doubles
    assert lib.saf3r_cosine_workspace_bytes(ctypes.byref(p), 64) == (64 * 172 + 172 * 172) * 8
    assert lib.saf3r_cosine_workspace_bytes(ctypes.byref(p), 0) == -1
    assert lib.saf3r_cosine_workspace_bytes(ctypes.byref(p), 4097) == -1
    assert lib.saf3r_cosine_workspace_bytes(None, 64) == -1
    cap = lib.saf3r_index_capacity
    # frames of 1374 tokens: a key block counts under the frame of its first
    # token, so frames hold 22 or 21 blocks (8 frames, 172 blocks)
    assert cap(ctypes.byref(p), B.head_table([(B.COSINE_TOPK, 1), (0, 0)])) == 8
    assert cap(ctypes.byref(p), B.head_table([(B.COSINE_TOPK, 2), (0, 0)])) == 16
    assert cap(ctypes.byref(p), B.head_table([(B.COSINE_TOPK, 64), (0, 0)])) == 172
    assert cap(ctypes.byref(p), B.head_table([(B.COSINE_TOPK, 65), (0, 0)])) == -5
    assert cap(ctypes.byref(p), B.head_table([(B.COSINE_TOPK, 0), (0, 0)])) == -5
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    t = B.head_table([(B.COSINE_TOPK, 2), (0, 0)])
    need = lib.saf3r_cosine_workspace_bytes(ctypes.byref(p), 64)
    sel = lib.saf3r_cosine_select
    assert sel(ctypes.byref(p), t, None, 64, fake, need, fake, fake, 16, None) == -1
    assert sel(ctypes.byref(p), t, fake, 0, fake, need, fake, fake, 16, None) == -1
    assert sel(ctypes.byref(p), t, fake, 64, fake, need - 8, fake, fake, 16, None) == -3
    assert sel(ctypes.byref(p), t, fake, 64, fake, need, fake, fake, 15, None) == -3


def test_nmse_entry_points_validate_before_launch(B):
    lib = B.load()
    p = _p(B, heads=3, frames=8, T=1374)
    # 128 (numerator, denominator) float64 pairs per head
    need = lib.saf3r_nmse_workspace_bytes(ctypes.byref(p))
    assert need == 3 * 128 * 16
    assert lib.saf3r_nmse_workspace_bytes(None) == -1
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first
    nm = lib.saf3r_nmse
    assert nm(ctypes.byref(p), None, fake, fake, need, fake, None) == -1
    assert nm(ctypes.byref(p), fake, fake, None, need, fake, None) == -1
    assert nm(ctypes.byref(p), fake, fake, fake, need, None, None) == -1
    assert nm(ctypes.byref(p), fake, fake, fake, need - 16, fake, None) == -3


def test_skip_heads_are_accepted_and_need_nothing(B):
    lib = B.load()
    cap = lib.saf3r_index_capacity
    p = _p(B, heads=3, frames=8, T=1374)
    assert cap(ctypes.byref(p), B.head_table([(B.SKIP, 0)] * 3)) == 1
    assert cap(ctypes.byref(p), B.head_table([(B.SKIP, 99), (2, 13), (B.SKIP, -4)])) == 13
    fake = ctypes.c_void_p(0x1000)
    # a table of SKIP and DENSE heads needs no lists: a missing output fails first
    t = B.head_table([(B.SKIP, 0), (0, 0), (B.SKIP, 0)])
    assert lib.saf3r_sparse_attention(ctypes.byref(p), t, fake, fake, fake, None, None, 0,
                                      None, None, None, 0, None) == -1


def test_missing_library_fails_loudly(B, tmp_path, monkeypatch):
    """Without the built library every entry of the binding raises; nothing
    falls back to another implementation."""
    monkeypatch.setattr(B, "_LIB", None)
    missing = str(tmp_path / "libsaf3r.so")
    with pytest.raises(RuntimeError, match="missing"):
        B.load(missing)
    monkeypatch.setattr(B, "LIB_PATH", missing)
    monkeypatch.setattr(B.load, "__defaults__", (missing,))
    with pytest.raises(RuntimeError, match="missing"):
        B.index_capacity([(B.TOPK, 4)], 2, 100)
    with pytest.raises(RuntimeError, match="missing"):
        B.attention_workspace_bytes([(B.TOPK, 4)], 2, 100)


def test_misaligned_pointers_are_rejected(B):
    """Every pointer the header requires to be aligned is checked before any
    launch: 16 bytes for Q/K/V/O, q_pooled, the NMSE inputs and workspaces;
    8 for k_pooled, scores and nmse_out; 4 for lists, counts and lse."""
    lib = B.load()
    p = _p(B, heads=2, frames=2, T=100)  # nb = 4
    t = B.head_table([(B.FRAME_LOCAL, 0), (B.TOPK, 2)])
    ok = ctypes.c_void_p(0x1000)
    a8, a4, a2 = ctypes.c_void_p(0x1008), ctypes.c_void_p(0x1004), ctypes.c_void_p(0x1002)
    est = lib.saf3r_estimate_blocks
    for args in ((a8, ok, ok, ok), (ok, a8, ok, ok), (ok, ok, a8, ok), (ok, ok, ok, a4)):
        assert est(ctypes.byref(p), t, *args, None) == -1, args
    sel = lib.saf3r_select_blocks
    need = lib.saf3r_select_workspace_bytes(ctypes.byref(p), t)
    for args in ((a4, ok, ok, ok, None, None), (ok, a4, ok, ok, None, None),
                 (ok, ok, a2, ok, None, None), (ok, ok, ok, a2, None, None),
                 (ok, ok, ok, ok, a4, None), (ok, ok, ok, ok, None, a8)):
        qp, kp, idx, cnt, scores, ws = args
        assert sel(ctypes.byref(p), t, qp, kp, idx, cnt, 8, scores, ws, need, None) == -1, args
    att = lib.saf3r_sparse_attention
    for args in ((a8, ok, ok, ok, ok, ok, None), (ok, a8, ok, ok, ok, ok, None),
                 (ok, ok, a8, ok, ok, ok, None), (ok, ok, ok, ok, ok, a8, None),
                 (ok, ok, ok, a2, ok, ok, None), (ok, ok, ok, ok, a2, ok, None),
                 (ok, ok, ok, ok, ok, ok, a2)):
        q, k, v, idx, cnt, out, lse = args
        assert att(ctypes.byref(p), t, q, k, v, idx, cnt, 8, out, lse, None, 0, None) == -1, args
    assert att(ctypes.byref(p), t, ok, ok, ok, ok, ok, 8, ok, None, a8, 1 << 20, None) == -1
    ct = B.head_table([(B.COSINE_TOPK, 1), (B.DENSE, 0)])
    cneed = lib.saf3r_cosine_workspace_bytes(ctypes.byref(p), 64)
    cos = lib.saf3r_cosine_select
    for args in ((ctypes.c_void_p(0x1001), ok, ok, ok), (ok, a4, ok, ok), (ok, ok, a2, ok),
                 (ok, ok, ok, a2)):
        f, ws, idx, cnt = args
        assert cos(ctypes.byref(p), ct, f, 64, ws, cneed, idx, cnt, 8, None) == -1, args
    pf = _p(B, heads=2, frames=2, T=100, dtype=B.F32)
    assert cos(ctypes.byref(pf), ct, a2, 64, ok, cneed, ok, ok, 8, None) == -1  # fp32: 4 bytes
    nm = lib.saf3r_nmse
    nneed = lib.saf3r_nmse_workspace_bytes(ctypes.byref(p))
    for args in ((a8, ok, ok, ok), (ok, a8, ok, ok), (ok, ok, a8, ok), (ok, ok, ok, a4)):
        f, s, ws, o = args
        assert nm(ctypes.byref(p), f, s, ws, nneed, o, None) == -1, args


def test_nmse_noalloc_validates_before_launch(B):
    """The allocation-free NMSE entry point checks its arguments like
    saf3r_nmse before it touches the device."""
    lib = B.load()
    p = _p(B, heads=3, frames=8, T=1374)
    ok, a8, a4 = ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1008), ctypes.c_void_p(0x1004)
    nm = lib.saf3r_nmse_noalloc
    assert nm(None, ok, ok, ok, None) == -1
    assert nm(ctypes.byref(_p(B, heads=0)), ok, ok, ok, None) == -1
    assert nm(ctypes.byref(_p(B, heads=257)), ok, ok, ok, None) == -2
    assert nm(ctypes.byref(p), None, ok, ok, None) == -1
    assert nm(ctypes.byref(p), ok, None, ok, None) == -1
    assert nm(ctypes.byref(p), ok, ok, None, None) == -1
    assert nm(ctypes.byref(p), a8, ok, ok, None) == -1
    assert nm(ctypes.byref(p), ok, a8, ok, None) == -1
    assert nm(ctypes.byref(p), ok, ok, a4, None) == -1


def test_validate_index_checks_arguments_before_launch(B):
    """The list check validates like the other calls before it launches; a
    table without list heads needs no launch at all."""
    lib = B.load()
    p = _p(B, heads=3, frames=8, T=1374)  # nb = 172
    t = B.head_table([(B.TOPK, 12), (B.FRAME_LOCAL, 0), (B.DENSE, 0)])
    ok, a2 = ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1002)
    first = ctypes.c_int32(-7)
    v = lib.saf3r_validate_index
    assert v(None, t, ok, ok, 12, ok, ctypes.byref(first), None) == -1
    assert v(ctypes.byref(p), None, ok, ok, 12, ok, ctypes.byref(first), None) == -1
    assert v(ctypes.byref(_p(B, heads=3, head_dim=32)), t, ok, ok, 12, ok, None, None) == -2
    assert v(ctypes.byref(p), B.head_table([(B.TOPK, 173), (B.DENSE, 0), (B.DENSE, 0)]),
             ok, ok, 12, ok, None, None) == -5
    assert v(ctypes.byref(p), t, None, ok, 12, ok, None, None) == -1
    assert v(ctypes.byref(p), t, ok, None, 12, ok, None, None) == -1
    assert v(ctypes.byref(p), t, ok, ok, 12, None, None, None) == -1
    assert v(ctypes.byref(p), t, ok, ok, 0, ok, None, None) == -1
    assert v(ctypes.byref(p), t, a2, ok, 12, ok, None, None) == -1
    assert v(ctypes.byref(p), t, ok, a2, 12, ok, None, None) == -1
    assert v(ctypes.byref(p), t, ok, ok, 12, a2, None, None) == -1
    assert first.value == -7  # untouched by a call that fails validation
    # DENSE, STRIDE and SKIP heads have no lists: nothing to launch or read
    none = B.head_table([(B.DENSE, 0), (B.STRIDE, 3), (B.SKIP, 0)])
    assert v(ctypes.byref(p), none, ok, ok, 1, ok, None, None) == 0
    assert lib.saf3r_status_string(-6).decode().startswith("corrupt kept-block list")

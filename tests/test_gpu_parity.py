"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Small workloads are compared in full (every list, every output element);
the large ones on a seeded sample of query blocks per head, which the oracle
computes one by one from the same inputs (rows are independent, so a sampled
row checks exactly that row of the full-size launch)."""
import numpy as np
import pytest

import oracle as O
from tests import parity as PT
from workloads import WORKLOADS, Workload, make_qkv, make_table

pytestmark = pytest.mark.gpu


def _tols(w):
    return (PT.TOL_BF16, PT.LSE_TOL_BF16) if w.dtype == "bf16" else (PT.TOL_F32, PT.LSE_TOL_F32)


def _stride_blocks(n, stride):
    return -(-(-(-n // stride)) // 64)


def _rank(pattern, param, scores, i, T):
    """The oracle ranking a near-tie row of this head is checked against."""
    if scores is None:
        return None
    return PT.ranking(pattern, param, scores if pattern == O.GLOBAL_PROBE else scores[i], T)


def _full_check(P, w, q, k, v, table, want_scores=True):
    res = PT.gpu_layer(P, w, q, k, v, table, want_scores=want_scores)
    ref = O.run_layer(q, k, v, table, w.tokens_per_frame, w.dtype)
    tol, lse_tol = _tols(w)
    nb = w.nb
    cap = res["idx"].shape[2]
    near = 0
    for h, (pattern, param) in enumerate(table):
        if pattern in (O.TOPK, O.GLOBAL_PROBE):
            # pooled means: exact sums of bf16 in fp64, division correctly rounded
            np.testing.assert_allclose(res["q_pooled"][h], ref["q_pooled"][h], rtol=1e-15, atol=0)
            np.testing.assert_allclose(res["k_pooled"][h], ref["k_pooled"][h], rtol=1e-15, atol=0)
            if want_scores and pattern == O.TOPK:
                np.testing.assert_allclose(res["scores"][h], ref["scores"][h], rtol=1e-12, atol=1e-13)
            if want_scores and pattern == O.GLOBAL_PROBE:  # probe scores in row 0
                np.testing.assert_allclose(res["scores"][h][0], ref["scores"][h], rtol=1e-12, atol=1e-13)
        if pattern == O.STRIDE:
            assert np.all(res["cnt"][h] == _stride_blocks(w.tokens, param)), f"head {h}: stride count"
        else:
            for i in range(nb):
                status = PT.check_lists(res, h, i, pattern, ref["lists"][h][i], ref["margins"][h][i], nb, cap,
                                        rank=_rank(pattern, param, ref["scores"][h], i, w.tokens_per_frame))
                near += status == "near_tie"
        out_ref, lse_ref = ref["out"][h], ref["lse"][h]
        if near and pattern not in (O.DENSE, O.STRIDE):
            lists = [PT.gpu_list(res, h, i) for i in range(nb)]
            qh, kh, vh = (O.to_f64(x[h], w.dtype) for x in (q, k, v))
            out_ref, lse_ref = O.attend_head(qh, kh, vh, lists, 64)
        err = PT.max_abs(res["out"][h], out_ref)
        assert err <= tol, f"head {h} (pattern {pattern}): max abs error {err}"
        lerr = PT.max_abs(res["lse"][h], lse_ref)
        assert lerr <= lse_tol, f"head {h}: lse max abs error {lerr}"
    return res, ref, near


@pytest.mark.parametrize("name", ["S4xT261-f32", "S8xT1374-bf16"])
def test_full_layer_parity(gpu_lib, name):
    import paper_2607_03612_amd as P

    w = WORKLOADS[name]
    q, k, v = make_qkv(w)
    table = make_table(w)
    print(f"[parity] full {name} table={table}", flush=True)
    _, _, near = _full_check(P, w, q, k, v, table)
    print(f"[parity] {name}: near-ties {near}", flush=True)


def _sampled_check(P, w, layer, samples, seed):
    q, k, v = make_qkv(w, layer=layer)
    table = make_table(w, layer=layer)
    print(f"[parity] sampled {w.name} layer {layer} table={table}", flush=True)
    res = PT.gpu_layer(P, w, q, k, v, table, want_scores=False)
    tol, lse_tol = _tols(w)
    nb, n, T = w.nb, w.tokens, w.tokens_per_frame
    cap = res["idx"].shape[2]
    rows = PT.sample_blocks(nb, samples, seed)
    near = 0
    for h, (pattern, topk) in enumerate(table):
        qh, kh, vh = (O.to_f64(x[h], w.dtype) for x in (q, k, v))
        kbar = O.pool_blocks(kh, 64) if pattern == O.TOPK else None
        for i in rows:
            r = O.block_range(i, n, 64)
            rank = None
            if pattern == O.TOPK:
                qbar = O.pool_blocks(qh[r.start:r.stop], 64)
                srow = O.block_scores(qbar, kbar)[0]
                lst, margin = O.topk_row(srow, topk)
                rank = PT.ranking(pattern, topk, srow)
            elif pattern == O.FRAME_LOCAL:
                lst, margin = O.frame_local_row(i, n, T, 64), np.inf
            else:
                lst, margin = np.arange(nb), np.inf
            status = PT.check_lists(res, h, i, pattern, lst, margin, nb, cap, rank=rank)
            if status == "near_tie":
                near += 1
                lst = PT.gpu_list(res, h, i)
            out_ref, lse_ref = O.attend_block(qh, kh, vh, i, lst, 64)
            err = PT.max_abs(res["out"][h][r.start:r.stop], out_ref)
            assert err <= tol, f"head {h} block {i}: max abs error {err}"
            lerr = PT.max_abs(res["lse"][h][r.start:r.stop], lse_ref)
            assert lerr <= lse_tol, f"head {h} block {i}: lse error {lerr}"
    print(f"[parity] {w.name} layer {layer}: {len(rows)} blocks/head, near-ties {near}", flush=True)


@pytest.mark.parametrize("name,layer", [("S32xT1374-bf16", 0), ("S100xT1374-bf16", 0),
                                        ("S200xT1374-bf16-L24", 0), ("S200xT1374-bf16-L24", 17)])
def test_sampled_parity_large(gpu_lib, name, layer):
    import paper_2607_03612_amd as P

    _sampled_check(P, WORKLOADS[name], layer, samples=24, seed=layer + 1)


def test_stack_layers_in_sequence(gpu_lib):
    """Two layers of the 24-layer stack run back to back as bench.py runs the
    stack: one index buffer sized for the larger capacity and viewed per
    layer, one selection workspace and one attention workspace shared by
    both, the earlier layer's lists overwritten by the later one's. Layer 8
    (Top-K k = 125, not split) then layer 5 (k = 959, split, one dense head);
    sampled rows of both against the oracle."""
    import torch

    import paper_2607_03612_amd as P

    w = WORKLOADS["S200xT1374-bf16-L24"]
    S, T, H, nb, n = w.frames, w.tokens_per_frame, w.heads, w.nb, w.tokens
    layers = []
    for layer in (8, 5):
        q, k, v = make_qkv(w, layer=layer)
        table = make_table(w, layer=layer)
        layers.append((layer, q, k, v, table, P.index_capacity(table, S, T)))
    idx_buf = torch.empty(H * nb * max(x[5] for x in layers), dtype=torch.int32, device="cuda")
    cnt = torch.empty((H, nb), dtype=torch.int32, device="cuda")
    sel_ws = torch.empty(max(P.select_workspace_bytes(x[4], S, T) for x in layers) // 4,
                         dtype=torch.int32, device="cuda")
    att_ws = torch.empty(max(P.attention_workspace_bytes(x[4], S, T) for x in layers) // 4,
                         dtype=torch.int32, device="cuda")
    assert P.attention_workspace_bytes(layers[1][4], S, T) > 0 == P.attention_workspace_bytes(layers[0][4], S, T)
    for layer, q, k, v, table, cap in layers:
        print(f"[parity] stack layer {layer} table={table}", flush=True)
        tq, tk, tv = (PT.to_device(x, "bf16") for x in (q, k, v))
        qp, kp = P.estimate_blocks(tq, tk, table, S, T)
        idx = idx_buf[: H * nb * cap].view(H, nb, cap)
        P.select_blocks(qp, kp, table, S, T, cap, idx, cnt, workspace=sel_ws)
        out, lse = P.sparse_attention(tq, tk, tv, table, S, T, idx, cnt, want_lse=True,
                                      workspace=att_ws)
        torch.cuda.synchronize()
        rows = PT.sample_blocks(nb, 6, layer)
        idx_h, cnt_h = idx.cpu().numpy(), cnt.cpu().numpy()
        for h, (pattern, topk) in enumerate(table):
            spans = [O.block_range(i, n, 64) for i in rows]
            got = [PT.out_to_numpy(out[h, r.start:r.stop]) for r in spans]
            got_lse = [lse[h, r.start:r.stop].cpu().numpy().astype(np.float64) for r in spans]
            qh, kh, vh = (O.to_f64(x[h], "bf16") for x in (q, k, v))
            kbar = O.pool_blocks(kh, 64) if pattern == O.TOPK else None
            for r_i, i in enumerate(rows):
                r = O.block_range(i, n, 64)
                rank = None
                if pattern == O.TOPK:
                    srow = O.block_scores(O.pool_blocks(qh[r.start:r.stop], 64), kbar)[0]
                    lst, margin = O.topk_row(srow, topk)
                    rank = PT.ranking(pattern, topk, srow)
                elif pattern == O.FRAME_LOCAL:
                    lst, margin = O.frame_local_row(i, n, T, 64), np.inf
                else:
                    lst, margin = np.arange(nb), np.inf
                PT.check_lists({"idx": idx_h, "cnt": cnt_h}, h, i, pattern, lst, margin, nb,
                               idx_h.shape[2], rank=rank)
                if pattern != O.DENSE:
                    lst = idx_h[h, i, :int(cnt_h[h, i])]
                ref, ref_lse = O.attend_block(qh, kh, vh, i, lst, 64)
                assert PT.max_abs(got[r_i], ref) <= PT.TOL_BF16, (layer, h, i)
                assert PT.max_abs(got_lse[r_i], ref_lse) <= PT.LSE_TOL_BF16, (layer, h, i)
        del tq, tk, tv, out, lse


def test_maximum_size_sampled(gpu_lib):
    """The largest problem the library accepts: N = 1048576 tokens (16384
    blocks) in 8 frames of 131072 tokens, two Top-K heads (k = 164) and one
    frame-local head (2048-block frames). Top-K scoring then runs two rows
    per workgroup and the row-in-LDS selection path; sampled rows against
    the oracle."""
    import paper_2607_03612_amd as P

    import torch

    w = Workload("max-8x131072", 8, 131072, "bf16", ("fixed", 0, 1, 1), heads=3)
    assert w.tokens == 1 << 20 and w.nb == 16384
    _sampled_check(P, w, 0, samples=6, seed=11)
    # the single-launch selection (two score rows per workgroup at this size)
    # gives the same lists as the workspace path checked above
    q, k, _ = make_qkv(w)
    table = make_table(w)
    tq, tk = (PT.to_device(x, "bf16") for x in (q, k))
    qp, kp = P.estimate_blocks(tq, tk, table, w.frames, w.tokens_per_frame)
    got = []
    for ws in (None, PT.select_workspace(P, table, w, heads=1)):
        idx, cnt, _ = P.select_blocks(qp, kp, table, w.frames, w.tokens_per_frame, workspace=ws)
        torch.cuda.synchronize()
        got.append((idx[:2].cpu().numpy(), cnt.cpu().numpy()))  # the two Top-K heads
    assert np.array_equal(got[0][1], got[1][1]) and np.array_equal(got[0][0], got[1][0])


@pytest.mark.parametrize("name,layer", [("S4xT261-f32", 0), ("S8xT1374-bf16", 0),
                                        ("S32xT1374-bf16", 0), ("S100xT1374-bf16", 0),
                                        ("S200xT1374-bf16-L24", 3)])
def test_select_paths_agree(gpu_lib, name, layer):
    """The single-launch Top-K selection (score rows in LDS) and the
    two-launch one (scores in a workspace, one wave per row), with a full
    workspace and with room for one head only (heads in batches), give the
    same lists, counts and scores bit for bit. S200 (nb = 4294) takes the
    row-in-LDS variant of the second launch."""
    import torch

    import paper_2607_03612_amd as P

    w = WORKLOADS[name]
    q, k, _ = make_qkv(w, layer=layer)
    table = make_table(w, layer=layer)
    code = P.BF16 if w.dtype == "bf16" else P.F32
    tq, tk = (PT.to_device(x, w.dtype) for x in (q, k))
    qp, kp = P.estimate_blocks(tq, tk, table, w.frames, w.tokens_per_frame)
    small = w.nb <= 1024  # the full score matrix is only kept for small layers
    runs = []
    for ws in (None, PT.select_workspace(P, table, w), PT.select_workspace(P, table, w, heads=1)):
        cap = P.index_capacity(table, w.frames, w.tokens_per_frame, code)
        idx = torch.full((w.heads, w.nb, cap), -7, dtype=torch.int32, device="cuda")
        cnt = torch.full((w.heads, w.nb), -9, dtype=torch.int32, device="cuda")
        _, _, sc = P.select_blocks(qp, kp, table, w.frames, w.tokens_per_frame, cap, idx, cnt,
                                   want_scores=small, dtype=code, workspace=ws)
        torch.cuda.synchronize()
        runs.append((idx.cpu().numpy(), cnt.cpu().numpy(), None if sc is None else sc.cpu().numpy()))
    for idx, cnt, sc in runs[1:]:
        assert np.array_equal(cnt, runs[0][1])
        assert np.array_equal(idx, runs[0][0])
        if small:
            assert np.array_equal(sc.view(np.uint64), runs[0][2].view(np.uint64))


def test_split_attention_paths_agree(gpu_lib):
    """Top-K lists of 578 key blocks (of 4294) on the 274800-token layer run
    split into four key ranges (with a workspace) and unsplit (without). Each
    path is within the bf16 bounds of the exact result, rounding P to bf16
    against different running maxima, so the two agree within twice those
    bounds; and the split launch is deterministic. The split path's parity
    against the oracle is checked by the sampled S200 tests, which run it."""
    import torch

    import paper_2607_03612_amd as P

    w = WORKLOADS["S200xT1374-bf16-L24"]
    layer = 3
    q, k, v = make_qkv(w, layer=layer)
    table = make_table(w, layer=layer)
    assert max(t for p, t in table if p == O.TOPK) >= 512
    S, T = w.frames, w.tokens_per_frame
    tq, tk, tv = (PT.to_device(x, "bf16") for x in (q, k, v))
    del q, k, v
    qp, kp = P.estimate_blocks(tq, tk, table, S, T)
    idx, cnt, _ = P.select_blocks(qp, kp, table, S, T, workspace=PT.select_workspace(P, table, w))
    ws = PT.attention_workspace(P, table, w)
    assert P.attention_workspace_bytes(table, S, T) > 0
    print(f"[parity] split vs unsplit {w.name} layer {layer} table={table}", flush=True)
    base, base_lse = P.sparse_attention(tq, tk, tv, table, S, T, idx, cnt, want_lse=True)
    runs = [P.sparse_attention(tq, tk, tv, table, S, T, idx, cnt, want_lse=True, workspace=ws)
            for _ in range(2)]
    torch.cuda.synchronize()
    for a, b in zip(runs[0], runs[1]):
        assert torch.equal(a, b), "split launch not deterministic"
    out, lse = runs[0]
    err = float((out.float() - base.float()).abs().max())
    lerr = float((lse - base_lse).abs().max())
    print(f"[parity] split vs unsplit: out {err:.3e}, lse {lerr:.3e}", flush=True)
    assert err <= 2 * PT.TOL_BF16 and lerr <= 2 * PT.LSE_TOL_BF16


def test_split_attention_with_global_probe_and_topk(gpu_lib):
    """Split attention on lists the library selects: a Top-K head (k = 400)
    and a global-probe head (k = 450) of 4294 key blocks both qualify for
    the key-range split, next to a frame-local, a dense and a stride-9 head (its
    own launch) that do not; sampled rows against the oracle's lists and
    attention."""
    import paper_2607_03612_amd as P

    w = WORKLOADS["S200xT1374-bf16-L24"]
    nb, n, T = w.nb, w.tokens, w.tokens_per_frame
    q, k, v = make_qkv(w, heads=[0, 1, 2, 3, 4])
    table = [(O.TOPK, 400), (O.GLOBAL_PROBE, 450), (O.FRAME_LOCAL, 0), (O.DENSE, 0), (O.STRIDE, 9)]
    assert P.attention_workspace_bytes(table, w.frames, T) == 2 * 4 * nb * 16896
    res = PT.gpu_layer(P, w, q, k, v, table)
    cap = res["idx"].shape[2]
    rows = PT.sample_blocks(nb, 8, 21)
    for h, (pattern, param) in enumerate(table):
        qh, kh, vh = (O.to_f64(x[h], "bf16") for x in (q, k, v))
        if pattern == O.GLOBAL_PROBE:
            glist, gmargin, gscores = O.global_probe_row(qh, kh, param, 64)
        kbar = O.pool_blocks(kh, 64) if pattern == O.TOPK else None
        for i in rows:
            r = O.block_range(i, n, 64)
            rank = None
            if pattern == O.TOPK:
                srow = O.block_scores(O.pool_blocks(qh[r.start:r.stop], 64), kbar)[0]
                lst, margin = O.topk_row(srow, param)
                rank = PT.ranking(pattern, param, srow)
            elif pattern == O.GLOBAL_PROBE:
                lst, margin = glist, gmargin
                rank = PT.ranking(pattern, param, gscores)
            elif pattern == O.FRAME_LOCAL:
                lst, margin = O.frame_local_row(i, n, T, 64), np.inf
            elif pattern == O.STRIDE:
                assert res["cnt"][h, i] == _stride_blocks(n, param)
                ref, ref_lse = O.attend_tokens(qh, kh, vh, r, O.stride_keys(n, param))
                assert PT.max_abs(res["out"][h][r.start:r.stop], ref) <= PT.TOL_BF16, (h, i)
                assert PT.max_abs(res["lse"][h][r.start:r.stop], ref_lse) <= PT.LSE_TOL_BF16, (h, i)
                continue
            else:
                lst, margin = np.arange(nb), np.inf
            if PT.check_lists(res, h, i, pattern, lst, margin, nb, cap, rank=rank) == "near_tie":
                lst = PT.gpu_list(res, h, i)
            ref, ref_lse = O.attend_block(qh, kh, vh, i, lst, 64)
            assert PT.max_abs(res["out"][h][r.start:r.stop], ref) <= PT.TOL_BF16, (h, i)
            assert PT.max_abs(res["lse"][h][r.start:r.stop], ref_lse) <= PT.LSE_TOL_BF16, (h, i)


def test_split_attention_custom_lists(gpu_lib):
    """Split attention on caller lists that exercise its cases: rows that
    reach only the first of the four key ranges (empty items), one-block
    rows, lists on the range boundaries, the partial last block, an empty
    row (zero output, LSE -inf) and lists of every length. Sampled rows
    against the oracle, every row against the unsplit launch."""
    import torch

    import paper_2607_03612_amd as P

    w = Workload("split-8x32766", 8, 32766, "bf16", ("fixed", 0, 0, 50), heads=2)
    nb, n = w.nb, w.tokens
    assert nb == 4096 and n % 64 == 48
    table = [(O.TOPK, 512), (O.TOPK, 600)]
    cap = 600
    q, k, v = make_qkv(w)
    g = np.random.default_rng(3)
    idx = np.full((2, nb, cap), -1, np.int32)
    cnt = np.zeros((2, nb), np.int32)
    for h in range(2):
        for i in range(nb):
            if h == 0 and i % 2 == 0:
                lst = np.arange(0, 1024, 2)  # only the first of the four key ranges
            elif h == 0 and i % 4 == 1:
                lst = np.sort(g.choice(nb, size=int(g.integers(1, 513)), replace=False))
            else:
                lst = np.sort(g.choice(nb, size=int(g.integers(1, cap + 1)), replace=False))
            idx[h, i, :len(lst)] = lst
            cnt[h, i] = len(lst)
    special = {(0, 5): [], (0, 7): [nb - 1], (1, 9): [0], (1, 11): list(range(3200, 3424)),
               (1, 13): [1023, 1024, 2047, 2048, 3071, 3072, nb - 1]}
    for (h, i), lst in special.items():
        idx[h, i] = -1
        idx[h, i, :len(lst)] = lst
        cnt[h, i] = len(lst)
    tq, tk, tv = (PT.to_device(x, "bf16") for x in (q, k, v))
    ti, tc = torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda()
    ws = PT.attention_workspace(P, table, w)
    assert P.attention_workspace_bytes(table, w.frames, w.tokens_per_frame) == 2 * 4 * nb * 16896
    out, lse = P.sparse_attention(tq, tk, tv, table, w.frames, w.tokens_per_frame, ti, tc,
                                  want_lse=True, workspace=ws)
    base, base_lse = P.sparse_attention(tq, tk, tv, table, w.frames, w.tokens_per_frame, ti, tc,
                                        want_lse=True)
    torch.cuda.synchronize()
    out_h, lse_h = PT.out_to_numpy(out), lse.cpu().numpy().astype(np.float64)
    base_h, base_lse_h = PT.out_to_numpy(base), base_lse.cpu().numpy().astype(np.float64)
    # the empty row: zero output and LSE -inf on both paths
    r5 = O.block_range(5, n, 64)
    assert np.all(out_h[0][r5.start:r5.stop] == 0) and np.all(np.isneginf(lse_h[0][r5.start:r5.stop]))
    assert np.all(np.isneginf(base_lse_h[0][r5.start:r5.stop]))
    fin = np.isfinite(base_lse_h)
    assert np.array_equal(fin, np.isfinite(lse_h))
    assert PT.max_abs(out_h, base_h) <= 2 * PT.TOL_BF16  # both within the bound of the exact result
    assert PT.max_abs(lse_h[fin], base_lse_h[fin]) <= 2 * PT.LSE_TOL_BF16
    rows = sorted(set(PT.sample_blocks(nb, 16, 4)) | {0, 1, 2, 3, 7, 9, 11, 13})
    for h in range(2):
        qh, kh, vh = (O.to_f64(x[h], "bf16") for x in (q, k, v))
        for i in rows:
            if cnt[h, i] == 0:  # the empty row, checked above
                continue
            r = O.block_range(i, n, 64)
            ref, ref_lse = O.attend_block(qh, kh, vh, i, idx[h, i, :cnt[h, i]], 64)
            err = PT.max_abs(out_h[h][r.start:r.stop], ref)
            assert err <= PT.TOL_BF16, f"head {h} block {i}: max abs error {err}"
            lerr = PT.max_abs(lse_h[h][r.start:r.stop], ref_lse)
            assert lerr <= PT.LSE_TOL_BF16, f"head {h} block {i}: lse error {lerr}"


# ------------------------------------------------------------ edge cases

EDGE = [
    # (frames, tokens_per_frame, dtype): partial last block of 1 token, a
    # single partial block, frames aligned to blocks, one frame
    (1, 129, "bf16"), (2, 20, "f32"), (4, 128, "bf16"), (1, 300, "f32"), (3, 100, "bf16"),
    (5, 261, "f32"),
]


@pytest.mark.parametrize("frames,T,dtype", EDGE)
def test_edge_shapes(gpu_lib, frames, T, dtype):
    import paper_2607_03612_amd as P

    w = Workload(f"edge-{frames}x{T}-{dtype}", frames, T, dtype, ("fixed", 1, 1, 50), heads=4)
    q, k, v = make_qkv(w)
    nb = w.nb
    table = [(O.DENSE, 0), (O.FRAME_LOCAL, 0), (O.TOPK, max(1, nb // 2)), (O.TOPK, nb)]
    print(f"[parity] edge {w.name} nb={nb}", flush=True)
    _full_check(P, w, q, k, v, table)


def test_topk_all_blocks_equals_dense_bitwise(gpu_lib):
    import paper_2607_03612_amd as P

    w = Workload("eq-dense", 3, 261, "bf16", ("fixed", 1, 1, 50), heads=2)
    q, k, v = make_qkv(w)
    for x in (q, k, v):
        x[1] = x[0]  # both heads see the same inputs
    a = PT.gpu_layer(P, w, q, k, v, [(O.DENSE, 0), (O.TOPK, w.nb)])
    np.testing.assert_array_equal(a["out"][0], a["out"][1])
    np.testing.assert_array_equal(a["lse"][0], a["lse"][1])


def test_uniform_values_give_uniform_output(gpu_lib):
    import paper_2607_03612_amd as P

    w = WORKLOADS["S8xT1374-bf16"]
    q, k, _ = make_qkv(w)
    v = np.full_like(q, 0x3F80)  # bf16 1.0
    res = PT.gpu_layer(P, w, q, k, v, make_table(w))
    assert np.max(np.abs(res["out"] - 1.0)) <= 2 ** -7


def test_runs_are_deterministic(gpu_lib):
    import paper_2607_03612_amd as P

    w = WORKLOADS["S8xT1374-bf16"]
    q, k, v = make_qkv(w, seed=5)
    table = make_table(w)
    a = PT.gpu_layer(P, w, q, k, v, table)
    b = PT.gpu_layer(P, w, q, k, v, table)
    for key in ("idx", "cnt", "out", "lse", "q_pooled", "k_pooled"):
        np.testing.assert_array_equal(a[key], b[key])


def test_exact_ties_go_to_the_lower_block(gpu_lib):
    """Duplicate key blocks give bit-identical scores on both sides; the tie
    rule (lower index first) must then pick the same blocks."""
    import paper_2607_03612_amd as P

    w = Workload("ties", 2, 320, "bf16", ("fixed", 0, 0, 50), heads=1)
    q, k, v = make_qkv(w)
    for dst, src in ((3, 1), (7, 1), (8, 5), (9, 5)):
        k[0, dst * 64:(dst + 1) * 64] = k[0, src * 64:(src + 1) * 64]
    nb = w.nb
    for topk in range(1, nb + 1):
        table = [(O.TOPK, topk)]
        res = PT.gpu_layer(P, w, q, k, v, table, want_lse=False)
        ref = O.run_layer(q, k, v, table, w.tokens_per_frame, "bf16", with_attention=False)
        for i in range(nb):
            np.testing.assert_array_equal(PT.gpu_list(res, 0, i), ref["lists"][0][i])


# All-dense layers run the shared-tile kernel (four query blocks of a head per
# workgroup): one, two and three key blocks, partial last blocks, head counts
# whose last workgroup has blocks past the head's end, and layers of more than
# 64 blocks (checked on sampled query blocks).
@pytest.mark.parametrize("frames,tpf,heads", [(2, 700, 4), (1, 20, 3), (1, 100, 5), (1, 130, 1),
                                              (1, 1990, 9), (1, 4100, 16), (2, 2200, 16)])
def test_all_dense_table_is_the_dense_baseline(gpu_lib, frames, tpf, heads):
    import paper_2607_03612_amd as P

    w = Workload("dense", frames, tpf, "bf16", ("fixed", heads, 0, 0), heads=heads)
    print(f"all-dense S={frames} T={tpf} H={heads} nb={w.nb}", flush=True)
    q, k, v = make_qkv(w)
    table = [(O.DENSE, 0)] * heads
    tq, tk, tv = (PT.to_device(x, "bf16") for x in (q, k, v))
    out, lse = P.sparse_attention(tq, tk, tv, table, w.frames, w.tokens_per_frame, want_lse=True)
    out = PT.out_to_numpy(out)
    lse = lse.cpu().numpy().astype(np.float64)
    n, nb = w.tokens, w.nb
    blocks = range(nb) if nb <= 40 else sorted({0, 1, 2, nb // 2, nb - 2, nb - 1})
    for h in range(heads) if nb <= 40 else (0, heads // 2, heads - 1):
        qh, kh, vh = (O.to_f64(x[h], "bf16") for x in (q, k, v))
        rows = np.concatenate([np.arange(i * 64, min(i * 64 + 64, n)) for i in blocks])
        o_ref, l_ref = O.dense_attention(qh[rows], kh, vh)
        assert PT.max_abs(out[h][rows], o_ref) <= PT.TOL_BF16, (h,)
        assert PT.max_abs(lse[h][rows], l_ref) <= PT.LSE_TOL_BF16, (h,)


@pytest.mark.parametrize("frames,tpf,heads", [(1, 130, 2), (2, 700, 4)])
def test_all_dense_table_fp32(gpu_lib, frames, tpf, heads):
    """fp32 layers have no shared-tile kernel: an all-dense fp32 table runs the
    list kernel with every head flagged dense."""
    import paper_2607_03612_amd as P

    w = Workload("dense-f32", frames, tpf, "f32", ("fixed", heads, 0, 0), heads=heads)
    q, k, v = make_qkv(w)
    tq, tk, tv = (PT.to_device(x, "f32") for x in (q, k, v))
    out, lse = P.sparse_attention(tq, tk, tv, [(O.DENSE, 0)] * heads, frames, tpf, want_lse=True)
    out = PT.out_to_numpy(out)
    lse = lse.cpu().numpy().astype(np.float64)
    for h in range(heads):
        o_ref, l_ref = O.dense_attention(*(O.to_f64(x[h], "f32") for x in (q, k, v)))
        assert PT.max_abs(out[h], o_ref) <= PT.TOL_F32, h
        assert PT.max_abs(lse[h], l_ref) <= PT.LSE_TOL_F32, h


def test_all_dense_launch_over_a_subset_of_heads(gpu_lib):
    """DENSE heads with SKIP heads between them still make an all-dense launch
    (the shared-tile kernel over the listed heads only): the dense heads get
    the same bits as in an all-dense table, the SKIP heads keep their rows."""
    import torch

    import paper_2607_03612_amd as P

    w = Workload("dense-skip", 2, 700, "bf16", ("fixed", 5, 0, 0), heads=5)
    q, k, v = make_qkv(w, seed=3)
    tq, tk, tv = (PT.to_device(x, "bf16") for x in (q, k, v))
    ref, ref_lse = P.sparse_attention(tq, tk, tv, [(O.DENSE, 0)] * 5, w.frames, w.tokens_per_frame,
                                      want_lse=True)
    table = [(O.DENSE, 0), (P.SKIP, 0), (O.DENSE, 0), (P.SKIP, 0), (O.DENSE, 0)]
    out = torch.full_like(tq, 7.0)
    _, lse = P.sparse_attention(tq, tk, tv, table, w.frames, w.tokens_per_frame, out=out,
                                want_lse=True)
    torch.cuda.synchronize()
    for h in range(5):
        if h % 2 == 0:
            assert torch.equal(out[h], ref[h]) and torch.equal(lse[h], ref_lse[h]), h
        else:
            assert bool((out[h] == 7.0).all()), h


# ------------------------------------------ anchor, stride, global probe


def _all_classes_table(w):
    nb, n = w.nb, w.tokens
    return [(O.DENSE, 0), (O.FRAME_LOCAL, 0), (O.TOPK, max(1, nb // 8)), (O.ANCHOR, 0),
            (O.ANCHOR, w.frames - 1), (O.STRIDE, 1), (O.STRIDE, 2), (O.STRIDE, 7),
            (O.STRIDE, min(64, n)), (O.STRIDE, max(1, n - 1)), (O.GLOBAL_PROBE, max(1, nb // 4)),
            (O.GLOBAL_PROBE, nb)]


@pytest.mark.parametrize("frames,T,dtype", [(4, 261, "f32"), (8, 1374, "bf16"), (3, 100, "bf16"),
                                            (1, 129, "bf16"), (2, 20, "f32")])
def test_all_classes_full_parity(gpu_lib, frames, T, dtype):
    import paper_2607_03612_amd as P

    w = Workload(f"classes-{frames}x{T}-{dtype}", frames, T, dtype, ("fixed", 1, 1, 50), heads=12)
    q, k, v = make_qkv(w)
    table = _all_classes_table(w)
    print(f"[parity] all classes {w.name} nb={w.nb} table={table}", flush=True)
    _, _, near = _full_check(P, w, q, k, v, table)
    print(f"[parity] {w.name}: near-ties {near}", flush=True)


def test_maximum_head_count_full_parity(gpu_lib):
    """256 heads, the most the library accepts, cycling through every class
    on a small ragged layer (3 frames x 100 tokens): per-class launches,
    the cost ordering of the list heads and the head indices carried in
    the kernel arguments all run at their limits."""
    import paper_2607_03612_amd as P

    w = Workload("heads256-3x100-bf16", 3, 100, "bf16", ("fixed", 1, 1, 50), heads=256)
    q, k, v = make_qkv(w)
    base = _all_classes_table(w)
    table = [base[h % len(base)] for h in range(256)]
    _, _, near = _full_check(P, w, q, k, v, table, want_scores=False)
    print(f"[parity] {w.name}: near-ties {near}", flush=True)


@pytest.mark.parametrize("cls", ["topk1", "topk_nb", "frame_local", "dense", "anchor", "stride5",
                                 "global2"])
def test_single_head_each_class(gpu_lib, cls):
    """A one-head layer of each class (grids and head lists of length one),
    on a ragged bf16 layer (5 frames x 150 tokens, 12 blocks, last one
    partial), checked in full against the oracle."""
    import paper_2607_03612_amd as P

    w = Workload(f"one-{cls}", 5, 150, "bf16", ("fixed", 1, 0, 50), heads=1)
    spec = {"topk1": (O.TOPK, 1), "topk_nb": (O.TOPK, w.nb), "frame_local": (O.FRAME_LOCAL, 0),
            "dense": (O.DENSE, 0), "anchor": (O.ANCHOR, 2), "stride5": (O.STRIDE, 5),
            "global2": (O.GLOBAL_PROBE, 2)}[cls]
    q, k, v = make_qkv(w)
    _full_check(P, w, q, k, v, [spec])


def test_stride_one_equals_dense_bitwise(gpu_lib):
    import paper_2607_03612_amd as P

    w = Workload("stride-eq-dense", 3, 261, "bf16", ("fixed", 1, 1, 50), heads=2)
    q, k, v = make_qkv(w)
    for x in (q, k, v):
        x[1] = x[0]
    a = PT.gpu_layer(P, w, q, k, v, [(O.DENSE, 0), (O.STRIDE, 1)])
    np.testing.assert_array_equal(a["out"][0], a["out"][1])
    np.testing.assert_array_equal(a["lse"][0], a["lse"][1])


def test_global_probe_gives_every_query_block_one_list(gpu_lib):
    import paper_2607_03612_amd as P

    w = WORKLOADS["S32xT1374-bf16"]
    q, k, v = make_qkv(w)
    table = [(O.GLOBAL_PROBE, 69)] + [(O.DENSE, 0)] * 15
    res = PT.gpu_layer(P, w, q, k, v, table, want_lse=False)
    rows = res["idx"][0, :, :int(res["cnt"][0, 0])]
    assert np.all(res["cnt"][0] == 69) and np.all(rows == rows[0])
    qh, kh = O.to_f64(q[0], "bf16"), O.to_f64(k[0], "bf16")
    sel, margin, s = O.global_probe_row(qh, kh, 69, 64)
    PT.check_lists(res, 0, 0, O.GLOBAL_PROBE, sel, margin, w.nb, res["idx"].shape[2],
                   rank=PT.ranking(O.GLOBAL_PROBE, 69, s))


def test_equal_scores_keep_the_lowest_block_indices(gpu_lib):
    """Every key token equal: all block scores are the same float64 value, so
    the Top-K and global-probe selections reduce to the tie rule of the
    oracle's stable sort (lowest block indices first). This drives the Top-K
    kernel through its tie-bucket refinement over the whole row and the radix
    select through a single bucket at every digit."""
    import paper_2607_03612_amd as P

    w = Workload("ties-3x261", 3, 261, "bf16", ("fixed", 1, 1, 50), heads=3)
    q, k, v = make_qkv(w)
    k[:] = k[0, 0]  # one key vector for every head and token
    table = [(O.GLOBAL_PROBE, 5), (O.TOPK, 7), (O.TOPK, w.nb - 1)]
    res = PT.gpu_layer(P, w, q, k, v, table, want_lse=False)
    for h, kk in enumerate((5, 7, w.nb - 1)):
        assert np.all(res["cnt"][h] == kk), h
        np.testing.assert_array_equal(res["idx"][h, :, :kk], np.tile(np.arange(kk), (w.nb, 1)))


def test_equal_scores_long_rows(gpu_lib):
    """The same tie rule where each lane of the selection owns 68 key blocks
    (nb = 4200): the two-launch selection holds such rows in registers and
    the single launch reads them from LDS; both must keep the lowest block
    indices, through the tie refinement over bucket members in every slot."""
    import torch

    import paper_2607_03612_amd as P

    w = Workload("ties-2x134400", 2, 134400, "bf16", ("fixed", 0, 0, 50), heads=2)
    assert w.nb == 4200
    q, k, _ = make_qkv(w)
    k[:] = k[0, 0]
    table = [(O.TOPK, 7), (O.TOPK, w.nb - 1)]
    tq, tk = (PT.to_device(x, "bf16") for x in (q, k))
    qp, kp = P.estimate_blocks(tq, tk, table, w.frames, w.tokens_per_frame)
    for ws in (PT.select_workspace(P, table, w), None):
        idx, cnt, _ = P.select_blocks(qp, kp, table, w.frames, w.tokens_per_frame, workspace=ws)
        torch.cuda.synchronize()
        idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
        for h, kk in enumerate((7, w.nb - 1)):
            assert np.all(cnt[h] == kk), (h, ws is None)
            np.testing.assert_array_equal(idx[h, :, :kk], np.tile(np.arange(kk), (w.nb, 1)))


@pytest.mark.parametrize("stride", [8, 33])
def test_stride_sampled_parity_large(gpu_lib, stride):
    """The 137400-token layer with STRIDE heads, checked on sampled query
    blocks against the oracle's strided attention."""
    import paper_2607_03612_amd as P

    w = WORKLOADS["S100xT1374-bf16"]
    q, k, v = make_qkv(w)
    table = [(O.STRIDE, stride)] * 2 + [(O.DENSE, 0)] * 14
    tq, tk, tv = (PT.to_device(x, "bf16") for x in (q, k, v))
    out, lse = P.sparse_attention(tq, tk, tv, table, w.frames, w.tokens_per_frame, want_lse=True)
    out = PT.out_to_numpy(out)
    lse = lse.cpu().numpy().astype(np.float64)
    keys = O.stride_keys(w.tokens, stride)
    for h in range(2):
        qh, kh, vh = (O.to_f64(x[h], "bf16") for x in (q, k, v))
        for i in PT.sample_blocks(w.nb, 12, stride + h):
            r = O.block_range(i, w.tokens, 64)
            o_ref, l_ref = O.attend_tokens(qh, kh, vh, r, keys)
            assert PT.max_abs(out[h][r.start:r.stop], o_ref) <= PT.TOL_BF16, (h, i)
            assert PT.max_abs(lse[h][r.start:r.stop], l_ref) <= PT.LSE_TOL_BF16, (h, i)


# ------------------------------------------------------- cosine top-k


def _features(n, dim, frames, T, seed):
    """Synthetic per-token features: a per-frame shared direction plus noise,
    so similar frames share structure (stand-in for DINO patch features)."""
    g = np.random.default_rng(seed)
    base = g.standard_normal((frames, dim))
    f = np.repeat(base, T, axis=0)[:n] * 0.8 + g.standard_normal((n, dim))
    return f.astype(np.float32)


@pytest.mark.parametrize("frames,T,dtype,dim,shared", [(8, 1374, "bf16", 64, False),
                                                       (4, 261, "f32", 96, True),
                                                       (3, 100, "bf16", 33, False),
                                                       (1, 129, "f32", 8, True)])
def test_cosine_topk_lists_and_attention(gpu_lib, frames, T, dtype, dim, shared):
    """Cosine lists against the oracle, and attention over them. `shared`:
    heads 0 and 3 keep the same count per frame (one group, found once and
    written to both rows) and the group order differs from the head order."""
    import torch

    import paper_2607_03612_amd as P

    w = Workload(f"cos-{frames}x{T}-{dtype}", frames, T, dtype, ("fixed", 1, 1, 50), heads=4)
    q, k, v = make_qkv(w)
    f32 = _features(w.tokens, dim, frames, T, seed=frames + T)
    if dtype == "bf16":  # round to bf16 bits (nearest even), as the inputs are
        bits = f32.view(np.uint32)
        f_in = ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16).astype(np.uint16)
    else:
        f_in = f32
    f64 = O.to_f64(f_in, dtype)
    if shared:
        table = [(O.COSINE_TOPK, 3), (O.COSINE_TOPK, 1), (O.TOPK, max(1, w.nb // 4)), (O.COSINE_TOPK, 3)]
    else:
        table = [(O.COSINE_TOPK, 1), (O.COSINE_TOPK, 3), (O.TOPK, max(1, w.nb // 4)), (O.DENSE, 0)]
    tq, tk, tv = (PT.to_device(x, dtype) for x in (q, k, v))
    code = P.BF16 if dtype == "bf16" else P.F32
    cap = P.index_capacity(table, frames, T, code)
    idx = torch.full((4, w.nb, cap), -7, dtype=torch.int32, device="cuda")
    cnt = torch.zeros((4, w.nb), dtype=torch.int32, device="cuda")
    P.cosine_select(PT.to_device(f_in, dtype), table, frames, T, idx, cnt)
    # select_blocks afterwards leaves the cosine rows as they are (cached lists)
    qp, kp = P.estimate_blocks(tq, tk, table, frames, T)
    P.select_blocks(qp, kp, table, frames, T, cap, idx, cnt, dtype=code)
    out, lse = P.sparse_attention(tq, tk, tv, table, frames, T, idx, cnt, want_lse=True)
    torch.cuda.synchronize()
    res = {"idx": idx.cpu().numpy(), "cnt": cnt.cpu().numpy(), "out": PT.out_to_numpy(out),
           "lse": lse.cpu().numpy().astype(np.float64)}
    ref = O.run_layer(q, k, v, table, T, dtype, features=f64)
    tol, lse_tol = _tols(w)
    near = 0
    for h, (pattern, param) in enumerate(table):
        near_h = 0
        for i in range(w.nb):
            status = PT.check_lists(res, h, i, pattern, ref["lists"][h][i], ref["margins"][h][i], w.nb, cap,
                                    rank=_rank(pattern, param, ref["scores"][h], i, T))
            near_h += status == "near_tie"
        near += near_h
        out_ref, lse_ref = ref["out"][h], ref["lse"][h]
        if near_h:  # the oracle's attention over the GPU's (valid) lists
            qh, kh, vh = (O.to_f64(x[h], dtype) for x in (q, k, v))
            out_ref, lse_ref = O.attend_head(qh, kh, vh, [PT.gpu_list(res, h, i) for i in range(w.nb)], 64)
        assert PT.max_abs(res["out"][h], out_ref) <= tol, h
        assert PT.max_abs(res["lse"][h], lse_ref) <= lse_tol, h
    print(f"[parity] cosine {w.name}: near-ties {near}", flush=True)


@pytest.mark.parametrize("frames,T,ks", [(70, 261, (1, 4, 1)), (130, 130, (2, 1, 64))])
def test_cosine_lists_many_frames(gpu_lib, frames, T, ks):
    """Cosine lists only (no attention) with more frames than lanes: 70 and
    130 frames take two and three passes of 64 frames per wave; two heads
    share a count, a SKIP head keeps its rows, and k = 64 keeps every block
    of a frame."""
    import torch

    import paper_2607_03612_amd as P

    w = Workload(f"cosl-{frames}x{T}", frames, T, "f32", ("fixed", 1, 1, 50), heads=4)
    q, k, _ = make_qkv(w)
    f_in = _features(w.tokens, 16, frames, T, seed=frames)
    table = [(O.COSINE_TOPK, ks[0]), (O.COSINE_TOPK, ks[1]), (P.SKIP, 0), (O.COSINE_TOPK, ks[2])]
    cap = P.index_capacity(table, frames, T, P.F32)
    idx = torch.full((4, w.nb, cap), -7, dtype=torch.int32, device="cuda")
    cnt = torch.full((4, w.nb), -9, dtype=torch.int32, device="cuda")
    P.cosine_select(PT.to_device(f_in, "f32"), table, frames, T, idx, cnt)
    torch.cuda.synchronize()
    res = {"idx": idx.cpu().numpy(), "cnt": cnt.cpu().numpy()}
    assert (res["idx"][2] == -7).all() and (res["cnt"][2] == -9).all()
    cos_table = [t if t[0] != P.SKIP else (O.DENSE, 0) for t in table]
    ref = O.run_layer(q, k, k, cos_table, T, "f32", features=O.to_f64(f_in, "f32"),
                      with_attention=False)
    for h in (0, 1, 3):
        for i in range(w.nb):
            PT.check_lists(res, h, i, O.COSINE_TOPK, ref["lists"][h][i], ref["margins"][h][i],
                           w.nb, cap, rank=_rank(O.COSINE_TOPK, table[h][1], ref["scores"][h], i, T))


# ------------------------------------------------- NMSE and the profiler


@pytest.mark.parametrize("frames,T", [(3, 261), (7, 1374), (1, 40)])
def test_nmse_kernel_matches_oracle(gpu_lib, frames, T):
    """Eq. 1 per head against the oracle's float64 sum. The sizes cover one
    partial slice per head (N = 40), slices that do not divide the head
    (N = 783) and many full slices (N = 9618); the result is also the same
    bits on a second call (fixed reduction order)."""
    import paper_2607_03612_amd as P

    for dtype in ("bf16", "f32"):
        w = Workload(f"nmse-{dtype}", frames, T, dtype, ("fixed", 1, 1, 50), heads=3)
        a, b, _ = make_qkv(w, seed=3)
        ta, tb = PT.to_device(a, dtype), PT.to_device(b, dtype)
        got = P.nmse(ta, tb, w.frames, w.tokens_per_frame).cpu().numpy()
        for h in range(3):
            want = O.nmse(O.to_f64(a[h], dtype), O.to_f64(b[h], dtype))
            assert abs(got[h] - want) <= 1e-12 * want, (dtype, h, got[h], want)
        again = P.nmse(ta, tb, w.frames, w.tokens_per_frame).cpu().numpy()
        assert np.array_equal(got.view(np.uint64), again.view(np.uint64))
        assert np.all(P.nmse(ta, ta, w.frames, w.tokens_per_frame).cpu().numpy() == 0.0)


def test_profiler_matches_oracle_search(gpu_lib):
    """Errors and costs of every (configuration, head) against the oracle's
    NMSE of Eq. 1 and FLOP count, and the Eq. 2 choice where the errors of
    the two best eligible configurations are clearly apart."""
    import paper_2607_03612_amd as P
    from paper_2607_03612_amd import profiler

    w = Workload("profile", 4, 261, "bf16", ("fixed", 0, 0, 50), heads=4)
    calib = [make_qkv(w, seed=s) for s in (11, 12)]
    dev = [tuple(PT.to_device(x, "bf16") for x in qkv) for qkv in calib]
    nb = w.nb
    cands = [(O.TOPK, 1), (O.TOPK, 2), (O.TOPK, 3), (O.GLOBAL_PROBE, 2), (O.FRAME_LOCAL, 0),
             (O.ANCHOR, 0), (O.STRIDE, 10)]
    res = profiler.profile_heads(dev, w.frames, w.tokens_per_frame, cands, sigma=0.85)
    configs = res["configs"]
    assert configs[0] == (O.STRIDE, O.baseline_stride(0.85))
    H, n = w.heads, w.tokens
    err_ref = np.zeros((len(configs), H))
    cost_ref = np.zeros((len(configs), H))
    for q, k, v in calib:
        for c, (pattern, param) in enumerate(configs):
            ref = O.run_layer(q, k, v, [(pattern, param)] * H, w.tokens_per_frame, "bf16")
            for h in range(H):
                qh, kh, vh = (O.to_f64(x[h], "bf16") for x in (q, k, v))
                full, _ = O.dense_attention(qh, kh, vh)
                err_ref[c, h] += O.nmse(full, ref["out"][h]) / len(calib)
                if pattern == O.STRIDE:
                    cost_ref[c, h] += O.attention_flops(n, 64, 64, stride=param) / len(calib)
                else:
                    cost_ref[c, h] += O.attention_flops(n, 64, 64, ref["lists"][h]) / len(calib)
    # exact counts; a near-tie row may keep a different block (rtol covers it)
    np.testing.assert_allclose(res["costs"], cost_ref, rtol=1e-3, atol=0)
    # bf16 outputs on both sides of the GPU error: a few 1e-3 relative
    np.testing.assert_allclose(res["errors"], err_ref, rtol=3e-2, atol=1e-5)
    for h in range(H):
        want = O.progressive_substitution(err_ref[:, h], cost_ref[:, h])
        eligible = sorted(err_ref[c, h] for c in range(len(configs)) if cost_ref[c, h] <= cost_ref[0, h])
        if len(eligible) < 2 or eligible[1] - eligible[0] > 0.1 * eligible[0]:
            assert res["choice"][h] == want, (h, res["errors"][:, h], err_ref[:, h])
    print(f"[profile] choice {res['choice']} table {res['table']}", flush=True)


def test_skip_heads_split_a_layer_across_streams(gpu_lib):
    """Static heads on one stream and Top-K heads on another (the rest marked
    SKIP in each call) give the same lists and outputs as one call, and a
    SKIP head's output is left untouched."""
    import torch

    import paper_2607_03612_amd as P

    w = WORKLOADS["S8xT1374-bf16"]
    q, k, v = make_qkv(w, seed=2)
    table = make_table(w)
    S, T, H, nb = w.frames, w.tokens_per_frame, w.heads, w.nb
    tq, tk, tv = (PT.to_device(x, "bf16") for x in (q, k, v))
    cap = P.index_capacity(table, S, T)
    ref_out, ref_idx, ref_cnt = P.run_layer(tq, tk, tv, table, S, T)
    dyn = [(p, a) if p == P.TOPK else (P.SKIP, 0) for p, a in table]
    sta = [(P.SKIP, 0) if p == P.TOPK else (p, a) for p, a in table]
    qp = torch.zeros((H, nb, 64), dtype=torch.float64, device="cuda")
    kp = torch.zeros((H, 64, nb), dtype=torch.float64, device="cuda")
    idx = torch.full((H, nb, cap), -9, dtype=torch.int32, device="cuda")
    cnt = torch.full((H, nb), -9, dtype=torch.int32, device="cuda")
    out = torch.full_like(tq, 7.0)
    side = torch.cuda.Stream()
    fork = torch.cuda.Event()
    fork.record()
    side.wait_event(fork)
    with torch.cuda.stream(side):
        P.select_blocks(qp, kp, sta, S, T, cap, idx, cnt)
        P.sparse_attention(tq, tk, tv, sta, S, T, idx, cnt, out)
    P.estimate_blocks(tq, tk, dyn, S, T, qp, kp)
    P.select_blocks(qp, kp, dyn, S, T, cap, idx, cnt)
    P.sparse_attention(tq, tk, tv, dyn, S, T, idx, cnt, out)
    join = torch.cuda.Event()
    join.record(side)
    torch.cuda.current_stream().wait_event(join)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().float().numpy(), ref_out.cpu().float().numpy())
    np.testing.assert_array_equal(cnt.cpu().numpy(), ref_cnt.cpu().numpy())
    for h, (p, _) in enumerate(table):
        if p != P.DENSE:
            np.testing.assert_array_equal(idx[h].cpu().numpy(), ref_idx[h].cpu().numpy())
    # an all-SKIP call touches nothing
    before = out.clone()
    P.sparse_attention(tq, tk, tv, [(P.SKIP, 0)] * H, S, T, idx, cnt, out)
    torch.cuda.synchronize()
    assert torch.equal(before, out)


# ------------------------------------------- bounds of the tile loads


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_rows_past_the_last_token_stay_unread_and_unwritten(gpu_lib, dtype):
    """A partial last key block (N = 10992 = 171 * 64 + 48) in the last head:
    Q, K and V are views at the start of larger buffers whose bytes after the
    last head hold NaN, and O is a view whose trailing bytes hold a sentinel.
    The kernels bound every K/V tile load by the head's extent (the rows past
    N read as zeros), so every output is finite and within the oracle's
    bound, and the bytes after O are untouched. Dense, frame-local and Top-K
    heads all walk the partial block."""
    import torch

    import paper_2607_03612_amd as P

    w = Workload(f"pad-8x1374-{dtype}", 8, 1374, dtype, ("fixed", 1, 1, 25), heads=3)
    assert w.tokens % 64 == 48
    q, k, v = make_qkv(w)
    table = [(O.TOPK, 9), (O.FRAME_LOCAL, 0), (O.DENSE, 0)]
    H, N = w.heads, w.tokens
    pad = 2 * 64 * 64  # two blocks of rows after the last head
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    nan_bits = 0x7FC0 if dtype == "bf16" else 0x7FC00000

    def padded(x):
        dev = PT.to_device(x, dtype)
        big = torch.empty(H * N * 64 + pad, dtype=tdt, device="cuda")
        if dtype == "bf16":
            big.view(torch.int16).fill_(nan_bits)
        else:
            big.view(torch.int32).fill_(nan_bits)
        big[:H * N * 64].copy_(dev.reshape(-1))
        return big, big[:H * N * 64].view(H, N, 64)

    (_, tq), (_, tk), (_, tv) = padded(q), padded(k), padded(v)
    obig = torch.full((H * N * 64 + pad,), 7.0, dtype=tdt, device="cuda")
    out = obig[:H * N * 64].view(H, N, 64)
    code = P.BF16 if dtype == "bf16" else P.F32
    qp, kp = P.estimate_blocks(tq, tk, table, w.frames, w.tokens_per_frame)
    idx, cnt, _ = P.select_blocks(qp, kp, table, w.frames, w.tokens_per_frame, dtype=code)
    print(f"[parity] padded last head {dtype}", flush=True)
    P.sparse_attention(tq, tk, tv, table, w.frames, w.tokens_per_frame, idx, cnt, out=out)
    torch.cuda.synchronize()
    got = PT.out_to_numpy(out)
    assert PT.finite(got), "rows past the last token reached the output"
    assert bool((obig[H * N * 64:] == 7.0).all()), "a store went past the output"
    ref = O.run_layer(q, k, v, table, w.tokens_per_frame, dtype)
    tol = PT.TOL_BF16 if dtype == "bf16" else PT.TOL_F32
    res = {"idx": idx.cpu().numpy(), "cnt": cnt.cpu().numpy()}
    for h, (pattern, param) in enumerate(table):
        out_ref = ref["out"][h]
        if pattern != O.DENSE:  # the oracle over the GPU's lists (checked elsewhere)
            lists = [PT.gpu_list(res, h, i) for i in range(w.nb)]
            out_ref = O.attend_head(*(O.to_f64(x[h], dtype) for x in (q, k, v)), lists, 64)[0]
        assert PT.max_abs(got[h], out_ref) <= tol, (h, pattern)


def test_split_attention_on_cosine_heads(gpu_lib):
    """Cosine Top-K heads whose per-frame lists reach 400 and 600 key blocks
    (2 and 3 of each of 200 frames) on a 274800-token layer (4294 key
    blocks) run through the key-range split; sampled rows' lists against the
    oracle's per-frame selection and outputs against the oracle's attention."""
    import torch

    import paper_2607_03612_amd as P

    w = WORKLOADS["S200xT1374-bf16-L24"]
    S, T, nb, n = w.frames, w.tokens_per_frame, w.nb, w.tokens
    q, k, v = make_qkv(w, heads=[0, 1])
    table = [(O.COSINE_TOPK, 2), (O.COSINE_TOPK, 3)]
    assert P.attention_workspace_bytes(table, S, T) == 2 * 4 * nb * 16896
    f_in = _features(n, 16, S, T, seed=5)
    bits = f_in.view(np.uint32)
    f_in = ((bits + 0x7FFF + ((bits >> 16) & 1)) >> 16).astype(np.uint16)  # bf16, nearest even
    cap = P.index_capacity(table, S, T)
    assert cap == 600
    idx = torch.full((2, nb, cap), -7, dtype=torch.int32, device="cuda")
    cnt = torch.zeros((2, nb), dtype=torch.int32, device="cuda")
    print(f"[parity] cosine split {w.name}", flush=True)
    P.cosine_select(PT.to_device(f_in, "bf16"), table, S, T, idx, cnt)
    tq, tk, tv = (PT.to_device(x, "bf16") for x in (q, k, v))
    ws = PT.attention_workspace(P, table, w)
    out, lse = P.sparse_attention(tq, tk, tv, table, S, T, idx, cnt, want_lse=True, workspace=ws)
    torch.cuda.synchronize()
    res = {"idx": idx.cpu().numpy(), "cnt": cnt.cpu().numpy()}
    fb = O.cosine_block_features(O.to_f64(f_in, "bf16"), 64)
    rows = PT.sample_blocks(nb, 8, 77)
    for h, (pattern, param) in enumerate(table):
        qh, kh, vh = (O.to_f64(x[h], "bf16") for x in (q, k, v))
        for i in rows:
            sim_row = fb @ fb[i]
            lst, margin = O.cosine_topk_row(sim_row, param, T, 64)
            if PT.check_lists(res, h, i, pattern, lst, margin, nb, cap,
                              rank=PT.ranking(pattern, param, sim_row, T)) == "near_tie":
                lst = PT.gpu_list(res, h, i)
            r = O.block_range(i, n, 64)
            ref, ref_lse = O.attend_block(qh, kh, vh, i, lst, 64)
            assert PT.max_abs(PT.out_to_numpy(out[h, r.start:r.stop]), ref) <= PT.TOL_BF16, (h, i)
            got_lse = lse[h, r.start:r.stop].cpu().numpy().astype(np.float64)
            assert PT.max_abs(got_lse, ref_lse) <= PT.LSE_TOL_BF16, (h, i)


# ------------------------------------------------------------ list check


def test_validate_index_passes_library_lists_and_finds_each_corruption(gpu_lib):
    """saf3r_validate_index: the lists the library writes pass (every class);
    each kind of corruption planted in one row of a copy is reported at that
    row, the lowest of two bad rows wins, and rows of DENSE / STRIDE heads are
    never read."""
    import torch

    import paper_2607_03612_amd as P

    w = Workload("check", 8, 1374, "bf16", ("fixed", 0, 0, 0))
    S, T, nb = w.frames, w.tokens_per_frame, w.nb
    table = _all_classes_table(w)
    H = len(table)
    q, k, _ = make_qkv(w, heads=range(H))
    tq, tk = (PT.to_device(x, "bf16") for x in (q, k))
    qp, kp = P.estimate_blocks(tq, tk, table, S, T)
    idx, cnt, _ = P.select_blocks(qp, kp, table, S, T)
    cap = idx.shape[2]
    assert P.validate_index(idx, cnt, table, S, T) is None

    topk = next(h for h, (p, _) in enumerate(table) if p == O.TOPK)
    fl = next(h for h, (p, _) in enumerate(table) if p == O.FRAME_LOCAL)
    row = 37
    k_top = table[topk][1]
    assert k_top < cap  # the Top-K rows carry padding

    def planted(h, i, fn):
        bi, bc = idx.clone(), cnt.clone()
        fn(bi[h, i], bc[h])
        return P.validate_index(bi, bc, table, S, T)

    def swap(r, c):
        r[[1, 2]] = r[[2, 1]]

    cases = {
        "unsorted": swap,
        "repeat": lambda r, c: r.__setitem__(1, r[0]),
        "negative": lambda r, c: r.__setitem__(0, -2),
        "past nb": lambda r, c: r.__setitem__(int(c[row]) - 1, nb),
        "padding": lambda r, c: r.__setitem__(cap - 1, 5),
        "count above cap": lambda r, c: c.__setitem__(row, cap + 1),
        "negative count": lambda r, c: c.__setitem__(row, -1),
    }
    for name, fn in cases.items():
        assert planted(topk, row, fn) == (topk, row), name
        assert planted(fl, row, fn) == (fl, row), name
    # Top-K keeps exactly k: one entry short is reported even when well formed
    assert planted(topk, row, lambda r, c: (c.__setitem__(row, k_top - 1),
                                            r.__setitem__(k_top - 1, -1))) == (topk, row)
    # two bad rows: the lowest (h * nb + i) is reported
    bi = idx.clone()
    bi[fl, 100, 0] = -2
    bi[topk, 5, 0] = nb + 3
    assert P.validate_index(bi, cnt, table, S, T) == (min(fl, topk), 100 if fl < topk else 5)
    # DENSE and STRIDE rows are not read, whatever they hold
    bi, bc = idx.clone(), cnt.clone()
    for h, (p, _) in enumerate(table):
        if p in (O.DENSE, O.STRIDE):
            bi[h].fill_(-9)
            bc[h].fill_(-9)
    assert P.validate_index(bi, bc, table, S, T) is None
    torch.cuda.synchronize()

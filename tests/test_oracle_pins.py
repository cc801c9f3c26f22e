"""Pins of the fp64 oracle against facts that do not come from the oracle.

Each pin checks an oracle function against a brute-force definition, a
library routine, a closed form or a hand-worked fixture, chosen so that a
plausible slip (a dropped term, a wrong scale, a transposed operand, an
off-by-one frame range, a reversed tie-break) fails at least one of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ---------------------------------------------------------------- inputs


def test_bf16_widening_known_bit_patterns():
    bits = np.array([0x3F80, 0xC000, 0x3FC0, 0x0000, 0x8000, 0x0001, 0x7F7F, 0x4049], np.uint16)
    want = [1.0, -2.0, 1.5, 0.0, -0.0, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127, 3.140625]
    got = O.to_f64(bits, "bf16")
    assert got.dtype == np.float64
    assert list(got) == want
    assert math.copysign(1.0, got[4]) == -1.0


def test_f32_widening_is_exact():
    x = np.array([0.1, -3.5e-20, 1e30], np.float32)
    assert list(O.to_f64(x, "f32")) == [float(v) for v in x]


# ------------------------------------------------- pooling + block scores


def _bruteforce_tile_means(q, k, block):
    """Mean of S = QK^T/sqrt(D) over each (query block, key block) tile,
    written with plain loops over tokens."""
    n, d = len(q), len(q[0])
    nb = (n + block - 1) // block
    out = [[0.0] * nb for _ in range(nb)]
    for i in range(nb):
        for j in range(nb):
            ti = range(i * block, min(n, (i + 1) * block))
            tj = range(j * block, min(n, (j + 1) * block))
            acc = 0.0
            for t in ti:
                for u in tj:
                    acc += sum(q[t][e] * k[u][e] for e in range(d)) / math.sqrt(d)
            out[i][j] = acc / (len(ti) * len(tj))
    return np.array(out)


@pytest.mark.parametrize("n,block,d", [(11, 4, 5), (8, 4, 3), (13, 13, 4), (9, 2, 6)])
def test_pooled_scores_equal_tile_mean_of_presoftmax_scores(n, block, d):
    q, k = _rand((n, d), 1), _rand((n, d), 2) * 3.0
    want = _bruteforce_tile_means(q.tolist(), k.tolist(), block)
    got = O.block_scores(O.pool_blocks(q, block), O.pool_blocks(k, block))
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    # not symmetric in (q, k): a transposed operand would fail
    if got.shape[0] > 1:
        assert not np.allclose(got, got.T)


def test_partial_last_block_divides_by_its_own_count():
    x = _rand((129, 64), 3)
    p = O.pool_blocks(x, 64)
    assert p.shape == (3, 64)
    np.testing.assert_array_equal(p[2], x[128])
    np.testing.assert_allclose(p[0], x[:64].mean(axis=0), rtol=0, atol=1e-15)


def test_global_probe_reproduces_column_mean_ranking():
    """The paper's identity (Sec. 4.3): ranking keys by the column mean of S
    equals ranking them by the single probe mean(q) K^T / sqrt(D)."""
    n, d = 40, 8
    q, k = _rand((n, d), 4), _rand((n, d), 5)
    s = [[sum(q[t, e] * k[u, e] for e in range(d)) / math.sqrt(d) for u in range(n)] for t in range(n)]
    colmean = np.array([sum(s[t][u] for t in range(n)) / n for u in range(n)])
    probe = O.block_scores(O.pool_blocks(q, n), O.pool_blocks(k, 1))[0]
    np.testing.assert_allclose(probe, colmean, rtol=1e-12, atol=1e-12)
    assert list(np.argsort(-probe, kind="stable")) == list(np.argsort(-colmean, kind="stable"))


# ---------------------------------------------------------------- top-k


def _bruteforce_topk(scores, k):
    """Among all k-subsets with the largest score sum, the lexicographically
    smallest sorted index tuple."""
    best = None
    for sub in itertools.combinations(range(len(scores)), k):
        key = (-sum(scores[j] for j in sub), sub)
        best = key if best is None or key < best else best
    return list(best[1])


@pytest.mark.parametrize("seed", range(6))
def test_topk_matches_bruteforce_over_subsets(seed):
    g = np.random.default_rng(seed)
    nb = 8
    s = g.standard_normal(nb)
    if seed % 2:  # plant exact ties
        s[g.integers(0, nb, 3)] = s[0]
    for k in range(1, nb + 1):
        got, margin = O.topk_row(s, k)
        assert list(got) == _bruteforce_topk(s.tolist(), k)
        if k == nb:
            assert margin == math.inf


def test_topk_worked_examples():
    cases = json.load(open(os.path.join(GOLDEN, "topk_worked_example.json")))["cases"]
    for c in cases:
        got, margin = O.topk_row(np.array(c["scores"]), c["k"])
        assert list(got) == c["selected"]
        assert margin == (math.inf if c["margin"] is None else c["margin"])


def test_topk_all_blocks_is_dense_selection():
    s = _rand(9, 6)
    got, _ = O.topk_row(s, 9)
    assert list(got) == list(range(9))


# ---------------------------------------------------------- frame-local


def test_frame_local_hand_worked_example():
    g = json.load(open(os.path.join(GOLDEN, "frame_local_N300_T100_B64.json")))
    for i, want in enumerate(g["lists"]):
        got = O.frame_local_row(i, g["tokens"], g["tokens_per_frame"], g["block"])
        assert list(got) == want


def test_frame_local_single_frame_keeps_everything():
    n = 1044
    nb = O.num_blocks(n, 64)
    for i in range(nb):
        assert list(O.frame_local_row(i, n, n, 64)) == list(range(nb))


def test_frame_local_aligned_frames_are_block_diagonal():
    n, T = 4 * 128, 128
    for i in range(8):
        assert list(O.frame_local_row(i, n, T, 64)) == [2 * (i // 2), 2 * (i // 2) + 1]


# ------------------------------------------------------------ attention


def _sdpa_masked(q, k, v, mask):
    """Library softmax attention (torch, fp64, CPU) with a boolean token mask."""
    tq, tk, tv = (torch.from_numpy(np.ascontiguousarray(x))[None] for x in (q, k, v))
    out = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, attn_mask=torch.from_numpy(mask)[None])
    return out[0].numpy()


def _token_mask(lists, n, block):
    mask = np.zeros((n, n), bool)
    for i, kept in enumerate(lists):
        for j in kept:
            mask[i * block:min(n, (i + 1) * block), j * block:min(n, (j + 1) * block)] = True
    return mask


@pytest.mark.parametrize("n,block,d", [(23, 4, 8), (64 * 3 + 1, 64, 64)])
def test_sparse_attention_matches_library_with_token_mask(n, block, d):
    q, k, v = _rand((n, d), 7) * 2, _rand((n, d), 8) * 2, _rand((n, d), 9)
    nb = O.num_blocks(n, block)
    g = np.random.default_rng(10)
    lists = [np.sort(g.choice(nb, size=int(g.integers(1, nb + 1)), replace=False)) for _ in range(nb)]
    out, lse = O.attend_head(q, k, v, lists, block)
    mask = _token_mask(lists, n, block)
    np.testing.assert_allclose(out, _sdpa_masked(q, k, v, mask), rtol=1e-11, atol=1e-12)
    z = np.where(mask, (q @ k.T) / math.sqrt(d), -np.inf)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=1), rtol=1e-12, atol=1e-12)


def test_dense_attention_matches_library():
    q, k, v = _rand((50, 16), 11), _rand((50, 16), 12), _rand((50, 16), 13)
    out, lse = O.dense_attention(q, k, v)
    np.testing.assert_allclose(out, _sdpa_masked(q, k, v, np.ones((50, 50), bool)), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(lse, scipy.special.logsumexp((q @ k.T) / 4.0, axis=1), rtol=1e-12)


def test_all_blocks_kept_equals_dense():
    n, d = 150, 64
    q, k, v = _rand((n, d), 14), _rand((n, d), 15), _rand((n, d), 16)
    lists, _, _ = O.select_head(O.DENSE, 0, q, k, n, 64)
    out, lse = O.attend_head(q, k, v, lists, 64)
    dout, dlse = O.dense_attention(q, k, v)
    np.testing.assert_allclose(out, dout, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(lse, dlse, rtol=1e-12)
    lists_k, _, _ = O.select_head(O.TOPK, O.num_blocks(n, 64), q, k, n, 64)
    assert all(list(x) == list(range(3)) for x in lists_k)


def test_attention_normalisation_and_single_key():
    n, d = 70, 64
    q, k = _rand((n, d), 17) * 3, _rand((n, d), 18) * 3
    ones = np.ones((n, d))
    out, _ = O.attend_head(q, k, ones, [np.array([0]), np.array([0, 1])], 64)
    np.testing.assert_allclose(out, 1.0, rtol=0, atol=1e-14)
    # a kept block with a single token gives that token's value row
    v = _rand((n, d), 19)
    out1, lse1 = O.attend_block(q, k, v, 0, np.array([1]), 64)  # block 1 = tokens 64..69
    out2, _ = O.attend_block(q[:65], k[:65], v[:65], 0, np.array([1]), 64)  # block 1 = token 64
    np.testing.assert_allclose(out2, np.broadcast_to(v[64], out2.shape), rtol=0, atol=1e-14)
    assert out1.shape == (64, d) and np.all(np.isfinite(lse1))


# ---------------------------------------------------------------- NMSE


def test_nmse_closed_forms():
    o = _rand((30, 8), 20)
    assert O.nmse(o, o) == 0.0
    assert O.nmse(o, np.zeros_like(o)) == pytest.approx(1.0, abs=1e-15)
    assert O.nmse(o, 1.25 * o) == pytest.approx(0.0625, rel=1e-12)
    assert O.nmse(o, -o) == pytest.approx(4.0, rel=1e-12)


# --------------------------------------------------------- whole layer


def test_run_layer_on_a_tiny_workload_is_consistent():
    from workloads import FRAME_LOCAL, TOPK, DENSE

    H, n, d, T = 3, 200, 64, 70
    g = np.random.default_rng(21)
    q = g.standard_normal((H, n, d)).astype(np.float32)
    k = g.standard_normal((H, n, d)).astype(np.float32)
    v = g.standard_normal((H, n, d)).astype(np.float32)
    table = [(DENSE, 0), (FRAME_LOCAL, 0), (TOPK, 2)]
    res = O.run_layer(q, k, v, table, T, "f32")
    for h in range(H):
        qh, kh, vh = (x[h].astype(np.float64) for x in (q, k, v))
        mask = _token_mask(res["lists"][h], n, 64)
        np.testing.assert_allclose(res["out"][h], _sdpa_masked(qh, kh, vh, mask), rtol=1e-11, atol=1e-12)
    assert [len(x) for x in res["lists"][2]] == [2] * 4
    # frames of 70 tokens: block 0 = frame 0 (tokens 0..63); frame 0 reaches block 1
    assert list(res["lists"][1][0]) == [0, 1]


# ------------------------------------- anchor frame, global probe, stride


def test_anchor_row_matches_token_bruteforce():
    """Anchor-frame static pattern: the blocks holding a token of the anchor
    frame, written with a plain token loop."""
    for n, T, block in [(300, 100, 64), (257, 61, 16), (64, 64, 64), (130, 7, 8)]:
        frames = -(-n // T)
        for a in range(frames):
            want = sorted({t // block for t in range(n) if t // T == a})
            assert list(O.anchor_row(a, n, T, block)) == want


def test_anchor_hand_worked_example():
    # N=300, T=100, block 64: frame 1 is tokens 100..199 -> blocks 1 (64..127),
    # 2 (128..191) and 3 (192..255); frame 2 (200..299) -> blocks 3 and 4
    assert list(O.anchor_row(1, 300, 100, 64)) == [1, 2, 3]
    assert list(O.anchor_row(2, 300, 100, 64)) == [3, 4]
    assert list(O.anchor_row(0, 300, 100, 64)) == [0, 1]


def _bruteforce_column_mean_block_scores(q, k, block):
    """Sec. 4.3 by definition: S = QK^T/sqrt(D) in plain loops, its column mean
    over all queries, then averaged over the tokens of each key block."""
    n, d = len(q), len(q[0])
    col = [sum(sum(q[t][e] * k[u][e] for e in range(d)) / math.sqrt(d) for t in range(n)) / n
           for u in range(n)]
    nb = (n + block - 1) // block
    return [sum(col[u] for u in range(j * block, min(n, (j + 1) * block)))
            / len(range(j * block, min(n, (j + 1) * block))) for j in range(nb)]


@pytest.mark.parametrize("n,block,d,k", [(37, 8, 5, 2), (24, 4, 3, 6), (9, 9, 4, 1)])
def test_global_probe_row_matches_column_mean_definition(n, block, d, k):
    q, k_ = _rand((n, d), 21) + 0.5, _rand((n, d), 22) * 2.0
    want_scores = np.array(_bruteforce_column_mean_block_scores(q.tolist(), k_.tolist(), block))
    sel, margin, s = O.global_probe_row(q, k_, k, block)
    np.testing.assert_allclose(s, want_scores, rtol=1e-12, atol=1e-12)
    assert list(sel) == _bruteforce_topk(want_scores.tolist(), k)


def test_global_probe_differs_from_per_block_probe():
    """The global probe gives every query block one list; per-block probes
    (TOPK) generally differ, so a class mix-up would show."""
    n, d = 96, 8
    g = np.random.default_rng(23)
    q = g.standard_normal((n, d))
    q[:48] += 3.0 * g.standard_normal(d)   # two groups of queries that prefer
    q[48:] += 3.0 * g.standard_normal(d)   # different keys
    k = g.standard_normal((n, d)) * 2.0
    lists_g, _, _ = O.select_head(O.GLOBAL_PROBE, 2, q, k, 48, 16)
    lists_t, _, _ = O.select_head(O.TOPK, 2, q, k, 48, 16)
    assert all(list(x) == list(lists_g[0]) for x in lists_g)
    assert any(list(x) != list(lists_g[0]) for x in lists_t)


def test_stride_keys_and_fraction():
    assert list(O.stride_keys(10, 3)) == [0, 3, 6, 9]
    assert list(O.stride_keys(5, 1)) == [0, 1, 2, 3, 4]
    assert list(O.stride_keys(7, 7)) == [0]
    # kept fraction 1/s when s divides N (the #Keys column of the stride rows)
    for n, s_ in [(4096, 64), (4096, 32), (1374, 2)]:
        assert len(O.stride_keys(n, s_)) * s_ == n


@pytest.mark.parametrize("n,stride", [(50, 3), (64, 64), (33, 1), (40, 7)])
def test_stride_attention_matches_library_with_token_mask(n, stride):
    d = 8
    q, k, v = _rand((n, d), 31), _rand((n, d), 32) * 2.0, _rand((n, d), 33)
    out, lse = O.attend_stride(q, k, v, stride)
    mask = torch.zeros((n, n), dtype=torch.bool)
    mask[:, ::stride] = True
    tq, tk, tv = (torch.from_numpy(x)[None, None] for x in (q, k, v))
    want = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask[None, None])[0, 0]
    np.testing.assert_allclose(out, want.numpy(), rtol=1e-12, atol=1e-12)
    z = q @ k[::stride].T / math.sqrt(d)
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=1), rtol=1e-12, atol=1e-12)
    if stride == 1:
        dense_out, _ = O.dense_attention(q, k, v)
        np.testing.assert_allclose(out, dense_out, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------ cosine top-k


def _bruteforce_tile_cosine(f, block):
    n = len(f)
    nb = (n + block - 1) // block
    norm = [math.sqrt(sum(x * x for x in row)) for row in f]
    out = [[0.0] * nb for _ in range(nb)]
    for i in range(nb):
        for j in range(nb):
            ti = range(i * block, min(n, (i + 1) * block))
            tj = range(j * block, min(n, (j + 1) * block))
            acc = 0.0
            for t in ti:
                for u in tj:
                    acc += sum(f[t][e] * f[u][e] for e in range(len(f[0]))) / (norm[t] * norm[u])
            out[i][j] = acc / (len(ti) * len(tj))
    return np.array(out)


@pytest.mark.parametrize("n,block,d", [(23, 4, 6), (16, 8, 3), (10, 10, 5)])
def test_cosine_block_similarity_is_tile_mean_of_token_cosines(n, block, d):
    f = _rand((n, d), 41) + 0.3
    fb = O.cosine_block_features(f, block)
    np.testing.assert_allclose(fb @ fb.T, _bruteforce_tile_cosine(f.tolist(), block), rtol=1e-12, atol=1e-12)
    # unit tokens: a one-token block's feature has length 1
    one = O.cosine_block_features(f, 1)
    np.testing.assert_allclose(np.sum(one * one, axis=1), 1.0, rtol=1e-14)


@pytest.mark.parametrize("seed", range(4))
def test_cosine_topk_row_is_per_frame_bruteforce(seed):
    g = np.random.default_rng(50 + seed)
    T, block = 20, 4          # frames of 20 tokens, blocks of 4: block j is in frame (4j)//20
    nb = 15                   # N = 60 tokens, 3 frames of 5 blocks each
    sim = g.standard_normal(nb)
    if seed % 2:
        sim[[1, 3, 7]] = sim[0]  # planted ties
    for k in (1, 2, 5, 6):
        got, _ = O.cosine_topk_row(sim, k, T, block)
        want = []
        for f in range(3):
            js = [j for j in range(nb) if (block * j) // T == f]
            kk = min(k, len(js))
            want += [js[x] for x in _bruteforce_topk([sim[j] for j in js], kk)]
        assert list(got) == sorted(want)


def test_cosine_topk_frame_of_a_straddling_block():
    # T = 6, block = 4: block 1 holds tokens 4..7 (frames 0 and 1) and counts
    # under frame 0, the frame of its first token
    assert [O.block_frame(j, 6, 4) for j in range(5)] == [0, 0, 1, 2, 2]
    sim = np.array([0.1, 0.9, 0.5, 0.2, 0.3])
    got, margin = O.cosine_topk_row(sim, 1, 6, 4)
    assert list(got) == [1, 2, 4]
    assert margin == pytest.approx(min(0.9 - 0.1, 0.3 - 0.2))


# ------------------------------------------------ offline profiling (Eq. 1-2)


def test_attention_flops_counts_token_pairs():
    # lists: query block 0 (64 tokens) keeps blocks {0, 2}; block 1 keeps {1};
    # block 2 (partial: 20 tokens) keeps {0, 1, 2}; d = 8 -> 4 d = 32 per pair
    n, d, block = 148, 8, 64
    lists = [np.array([0, 2]), np.array([1]), np.array([0, 1, 2])]
    pairs = 64 * (64 + 20) + 64 * 64 + 20 * (64 + 64 + 20)
    assert O.attention_flops(n, d, block, lists) == 32 * pairs
    # stride: every query against ceil(n / s) keys
    assert O.attention_flops(10, d, block, stride=3) == 32 * 10 * 4
    # dense lists equal 4 d n^2
    dense = [np.arange(3)] * 3
    assert O.attention_flops(n, d, block, dense) == 4 * d * n * n


def test_progressive_substitution_follows_eq2():
    # base error 0.5 cost 10; candidate 2 is best but too costly; candidate 3
    # ties candidate 1 and comes later (no replacement on ties)
    errors = [0.5, 0.2, 0.05, 0.2, 0.3]
    costs = [10, 10, 11, 9, 8]
    assert O.progressive_substitution(errors, costs) == 1
    assert O.progressive_substitution([0.1, 0.2, 0.3], [5, 5, 5]) == 0  # base stays
    assert O.progressive_substitution([0.1, 0.0], [5, 6]) == 0          # over budget
    assert O.progressive_substitution([0.1, 0.0], [5, 5]) == 1
    # equals the constrained argmin with ties to the earlier entry
    g = np.random.default_rng(61)
    for _ in range(50):
        e = g.integers(0, 4, 8).astype(float)
        c = g.integers(0, 5, 8)
        ok = [i for i in range(8) if c[i] <= c[0]]
        assert O.progressive_substitution(e, c) == min(ok, key=lambda i: (e[i], i))


def test_baseline_stride_reaches_the_sparsity():
    assert O.baseline_stride(0.85) == 7   # keeps 1/7 = 14.3% of keys
    assert O.baseline_stride(0.5) == 2
    assert O.baseline_stride(0.0) == 1
    assert O.baseline_stride(0.75) == 4

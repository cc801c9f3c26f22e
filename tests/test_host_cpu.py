"""Host-side logic of the profiler (no GPU): the baseline stride, the FLOP
count of Eq. 2 and the progressive-substitution choice, each against the
oracle's own definition on many seeded cases."""
import numpy as np
import pytest

import oracle as O
from paper_2607_03612_amd import binding as B
from paper_2607_03612_amd import profiler


@pytest.mark.parametrize("sigma", [0.0, 0.5, 0.6, 0.75, 0.8, 0.85, 0.9, 0.95, 0.97, 0.99])
def test_baseline_stride_matches_oracle(sigma):
    assert profiler.baseline_stride(sigma) == O.baseline_stride(sigma)


def test_baseline_stride_rejects_out_of_range():
    for sigma in (-0.1, 1.0, 1.5):
        with pytest.raises(ValueError):
            profiler.baseline_stride(sigma)


@pytest.mark.parametrize("n", [40, 64, 129, 1044, 1374])
def test_attention_cost_matches_oracle_flops(n):
    g = np.random.default_rng(n)
    nb = -(-n // 64)
    assert profiler.attention_cost(B.DENSE, 0, n) == O.attention_flops(n, 64, 64, [range(nb)] * nb)
    for s in (1, 2, 7, n - 1, n):
        assert profiler.attention_cost(B.STRIDE, s, n) == O.attention_flops(n, 64, 64, stride=s)
    # lists of random lengths (the last block partial), padded with -1 up to cap
    cap = nb
    lists = [np.sort(g.choice(nb, size=g.integers(1, nb + 1), replace=False)) for _ in range(nb)]
    idx = np.full((nb, cap), -1, np.int32)
    cnt = np.zeros(nb, np.int32)
    for i, lst in enumerate(lists):
        idx[i, :len(lst)] = lst
        cnt[i] = len(lst)
    assert profiler.attention_cost(B.TOPK, 0, n, idx, cnt) == O.attention_flops(n, 64, 64, lists)


def test_choice_matches_progressive_substitution():
    g = np.random.default_rng(7)
    for _ in range(200):
        C, H = int(g.integers(1, 8)), int(g.integers(1, 5))
        # few distinct values, so that ties in error and cost are common
        errors = g.integers(0, 4, size=(C, H)).astype(float)
        costs = g.integers(0, 4, size=(C, H)).astype(float)
        got = profiler.choose(errors, costs)
        want = [O.progressive_substitution(errors[:, h], costs[:, h]) for h in range(H)]
        assert got == want


def test_bench_refuses_more_than_one_gpu():
    """bench.py runs on one GPU; asking for more exits with status 2 and says
    so, before anything touches a GPU."""
    import subprocess
    import sys
    from pathlib import Path

    root = Path(__file__).resolve().parents[1]
    r = subprocess.run([sys.executable, str(root / "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def _list_len(pattern, param, n, T, nb):
    """Longest list of a head's class, from the oracle's own definitions."""
    if pattern == B.FRAME_LOCAL:
        # the longest list is a block's that holds a frame boundary (its list
        # contains both frames' blocks, so every list of either frame), or the
        # first block when there is one frame
        rows = {0, nb - 1} | {min((f * T) // 64, nb - 1) for f in range(1, -(-n // T))}
        return max(len(O.frame_local_row(i, n, T, 64)) for i in sorted(rows))
    if pattern == B.ANCHOR:
        return len(O.anchor_row(param, n, T, 64))
    if pattern == B.COSINE_TOPK:
        sim = np.random.default_rng(0).standard_normal(nb)
        return len(O.cosine_topk_row(sim, param, T, 64)[0])
    return param  # TOPK, GLOBAL_PROBE


@pytest.mark.parametrize("frames,T", [(2, 25000), (64, 400), (8, 5000), (40, 700), (3, 13000),
                                     (2, 131072), (64, 4100)])
def test_capacity_and_attention_split_match_oracle_lists(frames, T):
    """The library's index capacity (longest list over list heads) and the
    attention split (4 key ranges of nb items each: for bf16 on layers of
    4096 or more key blocks, list heads whose lists can hold 384 or more key
    blocks; and list or dense heads walking at least 32 (bf16) or 8 (fp32)
    blocks per query block, more than twice the layer's list-and-dense work
    over 2048 wave slots) against list lengths from the oracle's class
    definitions, on seeded random tables."""
    import ctypes

    lib = B.load()
    n = frames * T
    nb = -(-n // 64)
    g = np.random.default_rng(frames * 100003 + T)
    classes = [B.DENSE, B.FRAME_LOCAL, B.TOPK, B.ANCHOR, B.STRIDE, B.GLOBAL_PROBE, B.COSINE_TOPK, B.SKIP]
    for trial in range(12):
        table = []
        for _ in range(8):
            c = int(g.choice(classes))
            param = {B.TOPK: int(g.integers(1, nb + 1)), B.GLOBAL_PROBE: int(g.integers(1, nb + 1)),
                     B.ANCHOR: int(g.integers(0, frames)), B.STRIDE: int(g.integers(1, n + 1)),
                     B.COSINE_TOPK: int(g.integers(1, 65))}.get(c, 0)
            table.append((c, param))
        listed = [(c, p) for c, p in table if c in (B.FRAME_LOCAL, B.TOPK, B.ANCHOR, B.GLOBAL_PROBE,
                                                   B.COSINE_TOPK)]
        lens = [_list_len(c, p, n, T, nb) for c, p in listed]
        for dtype in (B.BF16, B.F32):
            p = B.problem(len(table), frames, T, dtype)
            t = B.head_table(table)
            assert lib.saf3r_index_capacity(ctypes.byref(p), t) == max(lens + [1]), (table, lens)
            n_dense = sum(1 for c, _ in table if c == B.DENSE)
            work = nb * (sum(lens) + n_dense * nb)

            def splits(cost, listed):
                bf16 = dtype == B.BF16
                return (bf16 and listed and nb >= 4096 and cost >= 384) or \
                    (cost >= (32 if bf16 else 8) and cost * 2048 > 2 * work)

            n_split = sum(1 for x in lens if splits(x, True)) + n_dense * splits(nb, False)
            want = 4 * nb * 16896 * n_split
            assert lib.saf3r_attention_workspace_bytes(ctypes.byref(p), t) == want, (table, lens)

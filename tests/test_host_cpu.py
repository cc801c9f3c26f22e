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

"""Helpers shared by the GPU parity tests: upload, run through the C ABI,
compare against the oracle. Holds none of the method's arithmetic."""
import math

import numpy as np

NEAR_TIE = 1e-6          # selection must be exact where the oracle margin exceeds this
TOL_BF16 = 2e-2          # max-abs error of bf16 outputs against the fp64 oracle
TOL_F32 = 1e-4           # max-abs error of fp32 outputs against the fp64 oracle
# Log-sum-exp: both dtypes accumulate the 64 products of q.k in fp32 (unit
# roundoff 6e-8); with |q||k| up to ~200 on these inputs the score error is
# ~1e-5 typical and bounded by ~1e-4, which the log-sum-exp inherits. The bf16
# path normalises by the sum of the bf16-rounded P it multiplies V with, so
# its log-sum-exp also carries bf16's relative rounding of P (at most 2^-8).
LSE_TOL_BF16 = 2.0 ** -8 + 1e-4
LSE_TOL_F32 = 1e-4


def to_device(x, dtype):
    import torch

    if dtype == "bf16":
        return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(x).cuda()


def out_to_numpy(t):
    import torch

    return t.float().cpu().numpy().astype(np.float64) if t.dtype == torch.bfloat16 else \
        t.cpu().numpy().astype(np.float64)


def select_workspace(P, table, w, heads=None):
    """A device workspace for the two-launch Top-K selection: the full size,
    or the share of `heads` TOPK heads."""
    import torch

    code = P.BF16 if w.dtype == "bf16" else P.F32
    full = P.select_workspace_bytes(table, w.frames, w.tokens_per_frame, code)
    n_topk = sum(1 for p, _ in table if p == 2)
    nbytes = full if heads is None or n_topk == 0 else full // n_topk * heads
    return torch.empty(max(nbytes, 16) // 4, dtype=torch.int32, device="cuda")


def attention_workspace(P, table, w):
    """A device workspace with which the attention splits its long lists
    into key ranges (16 bytes when no head qualifies)."""
    import torch

    code = P.BF16 if w.dtype == "bf16" else P.F32
    nbytes = P.attention_workspace_bytes(table, w.frames, w.tokens_per_frame, code)
    return torch.empty(max(nbytes, 16) // 4, dtype=torch.int32, device="cuda")


def gpu_layer(P, w, q, k, v, table, want_scores=False, want_lse=True, workspace=True):
    """Runs estimate -> select -> attend through the binding; returns numpy
    results. `workspace`: the two-launch Top-K selection and the attention
    that splits long lists into key ranges (as bench.py runs them) or, when
    False, the single-launch selection and unsplit attention."""
    import torch

    tq, tk, tv = (to_device(x, w.dtype) for x in (q, k, v))
    qp, kp = P.estimate_blocks(tq, tk, table, w.frames, w.tokens_per_frame)
    code = P.BF16 if w.dtype == "bf16" else P.F32
    ws = select_workspace(P, table, w) if workspace else None
    idx, cnt, scores = P.select_blocks(qp, kp, table, w.frames, w.tokens_per_frame,
                                       want_scores=want_scores, dtype=code, workspace=ws)
    del ws
    aws = attention_workspace(P, table, w) if workspace else None
    out, lse = P.sparse_attention(tq, tk, tv, table, w.frames, w.tokens_per_frame, idx, cnt,
                                  want_lse=want_lse, workspace=aws)
    torch.cuda.synchronize()
    res = {
        "q_pooled": qp.cpu().numpy(), "k_pooled": kp.transpose(1, 2).cpu().numpy(),
        "idx": idx.cpu().numpy(), "cnt": cnt.cpu().numpy(),
        "out": out_to_numpy(out), "lse": None if lse is None else lse.cpu().numpy().astype(np.float64),
        "scores": None if scores is None else scores.cpu().numpy(),
    }
    return res


def gpu_list(res, h, i):
    c = int(res["cnt"][h, i])
    return res["idx"][h, i, :c]


def ranking(pattern, param, score_row, tokens_per_frame=None):
    """What a near-tie row's list is checked against: the oracle's score row
    of a TOPK head (its probe scores for a GLOBAL_PROBE head) with the kept
    count, or a COSINE_TOPK head's similarity row with the per-frame count.
    None for the classes whose lists are fixed (no ranking)."""
    if pattern in (2, 5):  # TOPK, GLOBAL_PROBE
        return ("topk", np.asarray(score_row, np.float64), int(param))
    if pattern == 6:  # COSINE_TOPK
        return ("cosine", np.asarray(score_row, np.float64), int(param), int(tokens_per_frame))
    return None


def valid_topk(got, scores, k, tol=NEAR_TIE):
    """True when the ascending, distinct blocks `got` are a top-k of `scores`
    up to `tol`: exactly k blocks, every kept score at least s_(k) - tol and
    every dropped score at most s_(k+1) + tol, with s_(r) the r-th largest
    oracle score."""
    got = np.asarray(got, np.int64)
    nb = len(scores)
    if len(got) != k or k < 1 or k > nb:
        return False
    ranked = np.sort(scores)[::-1]
    kept = np.zeros(nb, bool)
    kept[got] = True
    if scores[kept].min() < ranked[k - 1] - tol:
        return False
    return k == nb or scores[~kept].max() <= ranked[k] + tol


def valid_ranking(got, rank, block=64):
    """`valid_topk` for a TOPK / GLOBAL_PROBE row, or per frame for a
    COSINE_TOPK row (the frame's min(k, blocks) most similar blocks, a block
    counted under the frame of its first token)."""
    import oracle as O

    if rank[0] == "topk":
        return valid_topk(got, rank[1], rank[2])
    _, sim, k, T = rank
    frame = np.array([O.block_frame(j, T, block) for j in range(len(sim))])
    got = np.asarray(got, np.int64)
    for f in np.unique(frame):
        js = np.nonzero(frame == f)[0]
        mine = np.searchsorted(js, got[frame[got] == f])
        if not valid_topk(mine, sim[js], min(k, len(js))):
            return False
    return True


def check_lists(res, h, i, pattern, oracle_list, margin, nb, cap, rank=None):
    """Returns 'ok', 'near_tie' or raises AssertionError with the row named.

    Lists must equal the oracle's where its margin exceeds NEAR_TIE. A
    near-tie row must still be a valid top-k of the oracle's ranking `rank`
    (see `ranking`); its outputs are then compared with the oracle run on
    the GPU's own list."""
    c = int(res["cnt"][h, i])
    if pattern == 0:  # DENSE: count only, list not materialised
        assert c == nb, f"head {h} block {i}: dense count {c} != {nb}"
        return "ok"
    row = res["idx"][h, i]
    assert np.all(row[c:] == -1), f"head {h} block {i}: padding not -1"
    got = row[:c]
    assert np.all(np.diff(got) > 0), f"head {h} block {i}: list not strictly ascending"
    assert got.min() >= 0 and got.max() < nb
    if margin <= NEAR_TIE:
        assert rank is not None, f"head {h} block {i}: near-tie row checked without the oracle's ranking"
        assert c == len(oracle_list) and valid_ranking(got, rank), \
            f"head {h} block {i}: near-tie list {list(got)} is not a valid top-k (oracle {list(oracle_list)})"
        return "near_tie"
    assert c == len(oracle_list) and np.array_equal(got, oracle_list), \
        f"head {h} block {i}: gpu {list(got)} != oracle {list(oracle_list)} (margin {margin})"
    return "ok"


def max_abs(a, b):
    return float(np.max(np.abs(a - b))) if a.size else 0.0


def sample_blocks(nb, count, seed):
    """Seeded sample of query blocks that always includes the first and last."""
    g = np.random.default_rng(seed)
    pick = set(g.choice(nb, size=min(count, nb), replace=False).tolist())
    pick |= {0, nb - 1}
    return sorted(pick)


def finite(x):
    return bool(np.all(np.isfinite(x)))


__all__ = ["NEAR_TIE", "TOL_BF16", "TOL_F32", "gpu_layer", "attention_workspace", "check_lists", "max_abs",
           "sample_blocks", "to_device", "out_to_numpy", "gpu_list", "ranking", "valid_topk",
           "valid_ranking", "math"]

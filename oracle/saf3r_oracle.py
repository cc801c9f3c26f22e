"""Plain fp64 CPU oracle of the SAF3R online hot path.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import this module. The product path (the HIP library and
its Python binding) never calls it and must fail loudly when the HIP library
is missing.

It follows the paper (SAF3R: Dynamic Sparse Attention for Feed-Forward 3D
Reconstruction Transformers) step by step, in float64, with no blocking,
fusion or reordering beyond what the definitions state:

1. Pooling (Sec. 4.3, Query-Probe Top-K): the probe of a set of queries is
   their mean. Read per query block of ``block`` tokens (and likewise per key
   block) over the tokens the block actually holds.
2. Scores (Sec. 4.3): by linearity of the inner product, the mean of the
   pre-softmax scores ``S = Q K^T / sqrt(D)`` over a (query block, key block)
   tile equals the scaled inner product of the two pooled vectors.
3. Selection per head class (Sec. 4.1 kernels; the class comes from the
   offline profile of Sec. 4.2): DENSE keeps every key block, FRAME_LOCAL (the
   static kernel) keeps the key blocks that share a frame with the query
   block, ANCHOR (the static kernel's anchor-frame example) keeps the key
   blocks of one designated frame, TOPK (the query-probe kernel per query
   block) keeps the ``k`` best-scoring key blocks with ties broken towards the
   lower block index, GLOBAL_PROBE (the query-probe kernel as Sec. 4.3 states
   it) ranks key blocks by the single mean query of the whole sequence and
   gives every query block the same ``k`` blocks, STRIDE (the uniform sampling
   kernel) keeps every ``s``-th key token, COSINE_TOPK (the DINO Top-K kernel,
   block-wise, on caller-supplied features) keeps per frame the ``k`` key
   blocks whose features are most similar to the query block's.
4. Attention restricted to the kept keys (Sec. 4.1, Query-Probe Top-K kernel):
   softmax over the kept key tokens, renormalised over that set, times V.
5. NMSE (Sec. 4.2, Eq. 1) between full and sparse outputs, the attention
   cost Omega in floating-point operations, and the progressive-substitution
   choice of Eq. 2 (the offline head profiling).

Pins (checked by the CPU tests, not by this module): pooling+scores against
the brute-force tile mean of S; Top-K against brute force over all k-subsets;
frame-local and anchor lists against hand-worked examples and token loops;
the cosine block similarity against the brute-force tile mean of token
cosine similarities and the per-frame selection against per-frame subset
enumeration;
the global probe against the column mean of the full S computed by brute
force (the identity of Sec. 4.3); attention (block lists and strided keys)
against a library softmax attention with an explicit token mask; NMSE
against closed forms. Every function here is pinned.
"""
from __future__ import annotations

import math

import numpy as np

DENSE = 0
FRAME_LOCAL = 1
TOPK = 2
ANCHOR = 3
STRIDE = 4
GLOBAL_PROBE = 5
COSINE_TOPK = 6


# --------------------------------------------------------------------------
# inputs


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact widening to float64 of fp32 values or of bf16 bit patterns."""
    if dtype == "bf16":
        bits = np.ascontiguousarray(x, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64)
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    raise ValueError(dtype)


def num_blocks(n: int, block: int) -> int:
    return (n + block - 1) // block


def block_range(b: int, n: int, block: int) -> range:
    """Tokens held by block ``b``; the last block may hold fewer than ``block``."""
    return range(b * block, min((b + 1) * block, n))


# --------------------------------------------------------------------------
# 1-2. pooling and block scores (Sec. 4.3)


def pool_blocks(x: np.ndarray, block: int) -> np.ndarray:
    """Mean of the rows of each block: ``x [N, D]`` -> ``[nb, D]``.

    The probe of Sec. 4.3 is the mean of the queries; per block, the mean is
    over the tokens the block holds (a partial last block divides by its own
    count)."""
    n, d = x.shape
    nb = num_blocks(n, block)
    out = np.empty((nb, d), np.float64)
    for b in range(nb):
        r = block_range(b, n, block)
        out[b] = x[r.start:r.stop].sum(axis=0) / len(r)
    return out


def block_scores(q_pooled: np.ndarray, k_pooled: np.ndarray) -> np.ndarray:
    """``s[i, j] = qbar_i . kbar_j / sqrt(D)``: the mean of S over tile (i, j)."""
    d = q_pooled.shape[1]
    return (q_pooled @ k_pooled.T) / math.sqrt(d)


# --------------------------------------------------------------------------
# 3. selection (Sec. 4.1 kernels, Sec. 4.3 Top-K)


def frames_of_block(b: int, n: int, tokens_per_frame: int, block: int) -> set:
    return {t // tokens_per_frame for t in block_range(b, n, block)}


def frame_local_row(i: int, n: int, tokens_per_frame: int, block: int) -> np.ndarray:
    """Key blocks sharing at least one frame with query block ``i`` (static
    kernel, block granularity): the blocks that hold a token whose frame is
    one of the frames of block ``i``."""
    fi = np.array(sorted(frames_of_block(i, n, tokens_per_frame, block)))
    token_frame = np.arange(n) // tokens_per_frame
    token_block = np.arange(n) // block
    return np.unique(token_block[np.isin(token_frame, fi)]).astype(np.int64)


def topk_row(scores_row: np.ndarray, k: int):
    """The ``k`` best key blocks of one query block.

    Order: score descending, then block index ascending (stable), first ``k``
    taken. Returns (ascending indices, margin) where the margin is the gap
    between the k-th and (k+1)-th ranked scores (+inf when every block is
    kept)."""
    nb = scores_row.shape[0]
    order = np.lexsort((np.arange(nb), -scores_row))
    chosen = np.sort(order[:k])
    margin = math.inf if k >= nb else float(scores_row[order[k - 1]] - scores_row[order[k]])
    return chosen.astype(np.int64), margin


def anchor_row(anchor: int, n: int, tokens_per_frame: int, block: int) -> np.ndarray:
    """Key blocks of the anchor frame (static kernel, Sec. 4.1: all queries
    look at one chosen frame): the blocks that hold a token of frame
    ``anchor``. The same for every query block."""
    token_frame = np.arange(n) // tokens_per_frame
    token_block = np.arange(n) // block
    return np.unique(token_block[token_frame == anchor]).astype(np.int64)


def global_probe_row(q_head: np.ndarray, k_head: np.ndarray, k: int, block: int):
    """Query-probe Top-K as Sec. 4.3 states it: one probe per head, the mean
    of all N queries; key block ``j`` scores ``qbar . kbar_j / sqrt(D)`` (the
    mean of S over all queries and the keys of block ``j``) and the ``k`` best
    blocks are kept (ties to the lower index) for every query block.

    Returns (ascending indices, margin, probe scores)."""
    d = q_head.shape[1]
    qbar = q_head.sum(axis=0) / q_head.shape[0]
    s = (pool_blocks(k_head, block) @ qbar) / math.sqrt(d)
    sel, margin = topk_row(s, k)
    return sel, margin, s


def cosine_block_features(f: np.ndarray, block: int) -> np.ndarray:
    """Block-wise feature for the DINO Top-K kernel (Sec. 4.3, block-wise
    variant): every token's feature scaled to unit length, then averaged over
    the block. The dot product of two such means is the mean cosine
    similarity over the (query block, key block) tile of token pairs."""
    norms = np.sqrt(np.sum(f * f, axis=1, keepdims=True))
    return pool_blocks(f / norms, block)


def block_frame(j: int, tokens_per_frame: int, block: int) -> int:
    """Frame a key block is counted under for per-frame selection: the frame
    of its first token."""
    return (j * block) // tokens_per_frame


def cosine_topk_row(sim_row: np.ndarray, k: int, tokens_per_frame: int, block: int):
    """Per-frame Top-K (Sec. 4.1, DINO Top-K: the most similar keys from each
    frame): for every frame, the ``k`` key blocks of that frame with the
    highest similarity (ties to the lower index; all of the frame's blocks if
    it has at most ``k``). Returns (ascending indices, margin) where the
    margin is the smallest gap, over frames that drop a block, between the
    k-th and (k+1)-th ranked similarities."""
    nb = sim_row.shape[0]
    frame = np.array([block_frame(j, tokens_per_frame, block) for j in range(nb)])
    kept, margin = [], math.inf
    for f in np.unique(frame):
        js = np.nonzero(frame == f)[0]
        sel, m = topk_row(sim_row[js], min(k, len(js)))
        kept.extend(js[sel].tolist())
        margin = min(margin, m)
    return np.array(sorted(kept), dtype=np.int64), margin


def stride_keys(n: int, stride: int) -> np.ndarray:
    """Key tokens kept by the uniform sampling kernel (Sec. 4.1): every
    ``stride``-th token, starting at token 0."""
    if stride < 1:
        raise ValueError("stride must be >= 1")
    return np.arange(0, n, stride, dtype=np.int64)


def select_head(pattern: int, topk: int, q_head: np.ndarray, k_head: np.ndarray,
                tokens_per_frame: int, block: int, features: np.ndarray = None):
    """Kept key blocks of every query block of one head.

    ``topk`` is the class parameter: the kept block count (TOPK,
    GLOBAL_PROBE), the anchor frame (ANCHOR), the key stride (STRIDE) or the
    blocks kept per frame (COSINE_TOPK, which also takes the per-token
    ``features``).
    Returns (lists, margins, scores): ``lists[i]`` ascending int64 (None for
    STRIDE, which keeps tokens, not blocks), ``margins`` the Top-K margins
    (+inf for the other classes), ``scores`` the block score matrix of a TOPK
    head or the probe scores of a GLOBAL_PROBE head (None otherwise)."""
    n = q_head.shape[0]
    nb = num_blocks(n, block)
    margins = np.full(nb, math.inf)
    if pattern == DENSE:
        return [np.arange(nb, dtype=np.int64) for _ in range(nb)], margins, None
    if pattern == FRAME_LOCAL:
        return [frame_local_row(i, n, tokens_per_frame, block) for i in range(nb)], margins, None
    if pattern == TOPK:
        if not 1 <= topk <= nb:
            raise ValueError("topk out of range")
        s = block_scores(pool_blocks(q_head, block), pool_blocks(k_head, block))
        lists = []
        for i in range(nb):
            sel, margins[i] = topk_row(s[i], topk)
            lists.append(sel)
        return lists, margins, s
    if pattern == ANCHOR:
        frames = -(-n // tokens_per_frame)
        if not 0 <= topk < frames:
            raise ValueError("anchor frame out of range")
        row = anchor_row(topk, n, tokens_per_frame, block)
        return [row for _ in range(nb)], margins, None
    if pattern == GLOBAL_PROBE:
        if not 1 <= topk <= nb:
            raise ValueError("topk out of range")
        sel, margin, s = global_probe_row(q_head, k_head, topk, block)
        margins[:] = margin
        return [sel for _ in range(nb)], margins, s
    if pattern == COSINE_TOPK:
        if topk < 1 or features is None:
            raise ValueError("cosine top-k needs k >= 1 and features")
        fb = cosine_block_features(features, block)
        sim = fb @ fb.T
        lists = []
        for i in range(nb):
            sel, margins[i] = cosine_topk_row(sim[i], topk, tokens_per_frame, block)
            lists.append(sel)
        return lists, margins, sim
    if pattern == STRIDE:
        # token-level: no block list; attention uses stride_keys
        if not 1 <= topk <= n:
            raise ValueError("stride out of range")
        return None, margins, None
    raise ValueError(f"unknown pattern {pattern}")


# --------------------------------------------------------------------------
# 4. attention over the kept keys (Sec. 4.1)


def attend_block(q_head: np.ndarray, k_head: np.ndarray, v_head: np.ndarray, i: int,
                 kept: np.ndarray, block: int):
    """Output rows and log-sum-exp of query block ``i`` over the kept key blocks.

    Softmax of ``q . k / sqrt(D)`` over the union of the kept blocks' tokens,
    renormalised over that set, applied to V."""
    n, d = q_head.shape
    rows = block_range(i, n, block)
    if len(kept) == 0:
        raise ValueError("a query block must keep at least one key block")
    spans = [block_range(int(j), n, block) for j in kept]
    keys = np.concatenate([np.arange(r.start, r.stop) for r in spans])
    z =(q_head[rows.start:rows.stop] @ k_head[keys].T) / math.sqrt(d)
    zmax = z.max(axis=1, keepdims=True)
    e = np.exp(z - zmax)
    denom = e.sum(axis=1, keepdims=True)
    out = (e / denom) @ v_head[keys]
    lse = (zmax + np.log(denom))[:, 0]
    return out, lse


def attend_tokens(q_head: np.ndarray, k_head: np.ndarray, v_head: np.ndarray, rows: range,
                  keys: np.ndarray):
    """Output rows and log-sum-exp of the query tokens ``rows`` over the key
    tokens ``keys``: softmax of ``q . k / sqrt(D)`` over that set, times V."""
    d = q_head.shape[1]
    z = (q_head[rows.start:rows.stop] @ k_head[keys].T) / math.sqrt(d)
    zmax = z.max(axis=1, keepdims=True)
    e = np.exp(z - zmax)
    denom = e.sum(axis=1, keepdims=True)
    return (e / denom) @ v_head[keys], (zmax + np.log(denom))[:, 0]


def attend_stride(q_head, k_head, v_head, stride: int):
    """Every query over the uniformly sampled keys (Sec. 4.1)."""
    n, d = q_head.shape
    return attend_tokens(q_head, k_head, v_head, range(0, n), stride_keys(n, stride))


def attend_head(q_head, k_head, v_head, lists, block: int):
    n, d = q_head.shape
    out = np.empty((n, d), np.float64)
    lse = np.empty(n, np.float64)
    for i, kept in enumerate(lists):
        r = block_range(i, n, block)
        out[r.start:r.stop], lse[r.start:r.stop] = attend_block(q_head, k_head, v_head, i, kept, block)
    return out, lse


def dense_attention(q_head, k_head, v_head):
    """Full softmax attention of one head (the paper's "Full" reference)."""
    d = q_head.shape[1]
    z = (q_head @ k_head.T) / math.sqrt(d)
    zmax = z.max(axis=1, keepdims=True)
    e = np.exp(z - zmax)
    denom = e.sum(axis=1, keepdims=True)
    return (e / denom) @ v_head, (zmax + np.log(denom))[:, 0]


# --------------------------------------------------------------------------
# 5. quality report (Sec. 4.2, Eq. 1)


def nmse(o_full: np.ndarray, o_sparse: np.ndarray) -> float:
    """``||O_full - O_sparse||^2 / ||O_full||^2`` for one head and one input."""
    num = float(np.sum((o_full - o_sparse) ** 2))
    den = float(np.sum(o_full ** 2))
    return num / den


def attention_flops(n: int, d: int, block: int, lists=None, stride: int = 0) -> int:
    """Omega(c) of Eq. 2: floating-point operations of attention restricted
    to the kept keys, 4 d per (query token, kept key token) pair (the Q K^T
    and P V products). Pass the per-query-block lists, or ``stride`` for the
    uniform sampling kernel."""
    if stride:
        return 4 * d * n * len(stride_keys(n, stride))
    total = 0
    for i, kept in enumerate(lists):
        keys = sum(len(block_range(int(j), n, block)) for j in kept)
        total += 4 * d * len(block_range(i, n, block)) * keys
    return total


def progressive_substitution(errors, costs) -> int:
    """Eq. 2 by progressive substitution (Sec. 4.2): entry 0 is the baseline
    c_base; walking the candidates in order, the current choice is replaced
    whenever a candidate has a strictly lower error and a cost not above the
    baseline's. Returns the index of c*."""
    best = 0
    for c in range(1, len(errors)):
        if costs[c] <= costs[0] and errors[c] < errors[best]:
            best = c
    return best


def baseline_stride(sigma: float) -> int:
    """Stride of the uniform sampling baseline with sparsity at least sigma:
    the smallest s with 1 - 1/s >= sigma."""
    s = 1
    while 1.0 - 1.0 / s < sigma - 1e-12:
        s += 1
    return s


# --------------------------------------------------------------------------
# whole layer


def run_layer(q, k, v, table, tokens_per_frame: int, dtype: str, block: int = 64,
              heads=None, with_attention: bool = True, features=None):
    """The whole hot path for one layer.

    ``q, k, v``: ``[H, N, D]`` fp32 arrays or bf16 bit patterns; ``table``:
    per-head ``(pattern, param)``; ``features``: per-token features ``[N, Df]``
    (float64) for COSINE_TOPK heads. Returns a dict with per-head lists,
    margins, pooled vectors (Top-K heads), scores, outputs and log-sum-exps
    (float64)."""
    H = q.shape[0]
    heads = range(H) if heads is None else heads
    res = {"lists": {}, "margins": {}, "scores": {}, "q_pooled": {}, "k_pooled": {},
           "out": {}, "lse": {}}
    for h in heads:
        pattern, topk = table[h]
        qh, kh = to_f64(q[h], dtype), to_f64(k[h], dtype)
        lists, margins, s = select_head(pattern, topk, qh, kh, tokens_per_frame, block, features)
        res["lists"][h], res["margins"][h], res["scores"][h] = lists, margins, s
        if pattern in (TOPK, GLOBAL_PROBE):
            res["q_pooled"][h] = pool_blocks(qh, block)
            res["k_pooled"][h] = pool_blocks(kh, block)
        if with_attention:
            vh = to_f64(v[h], dtype)
            if pattern == STRIDE:
                res["out"][h], res["lse"][h] = attend_stride(qh, kh, vh, topk)
            else:
                res["out"][h], res["lse"][h] = attend_head(qh, kh, vh, lists, block)
    return res

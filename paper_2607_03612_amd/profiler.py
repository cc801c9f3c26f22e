"""Offline head profiling by progressive local substitution (Sec. 4.2).

For every head, the search starts from the uniform sampling kernel whose
sparsity is at least sigma (the baseline c_base), measures the approximation
cost E(c) of Eq. 1 for each candidate configuration on calibration inputs,
and keeps, in candidate order, any candidate with a strictly lower E whose
attention cost Omega(c) (floating-point operations) does not exceed the
baseline's (Eq. 2). Every attention output and every E is computed by the HIP
library (dense and sparse attention, selection, saf3r_nmse); this module only
orders the candidates, counts Omega from the kept lists, and keeps the
choice.
"""
from __future__ import annotations

import math

import numpy as np

from . import binding as B


def baseline_stride(sigma: float) -> int:
    """The smallest key stride s whose sparsity 1 - 1/s is at least sigma."""
    if not 0.0 <= sigma < 1.0:
        raise ValueError("sigma must lie in [0, 1)")
    s = max(1, math.ceil(1.0 / (1.0 - sigma) - 1e-9))
    while 1.0 - 1.0 / s < sigma - 1e-12:
        s += 1
    return s


def attention_cost(pattern: int, param: int, n: int, idx=None, cnt=None) -> np.ndarray:
    """Omega of Eq. 2 for one head: floating-point operations of its
    head's attention, 4 * 64 per (query token, kept key token) pair.
    ``idx [nb, cap]`` and ``cnt [nb]`` are the head's kept lists (host)."""
    nb = -(-n // B.BLOCK)
    sizes = np.full(nb, B.BLOCK, np.int64)
    sizes[-1] = n - (nb - 1) * B.BLOCK
    if pattern == B.DENSE:
        return 4 * B.HEAD_DIM * n * n
    if pattern == B.STRIDE:
        return 4 * B.HEAD_DIM * n * (-(-n // param))
    listed = np.arange(idx.shape[1])[None, :] < cnt[:, None]
    key_tokens = np.where(listed, sizes[np.clip(idx, 0, nb - 1)], 0).sum(axis=1)
    return int(4 * B.HEAD_DIM * np.sum(sizes * key_tokens))


def profile_heads(calib, frames: int, tokens_per_frame: int, candidates, sigma: float = 0.85,
                  features=None, stream=None):
    """Progressive substitution for every head.

    ``calib``: list of ``(q, k, v)`` device tensors ``[H, N, 64]`` (one per
    calibration input, same shape and dtype); ``candidates``: list of
    ``(pattern, param)`` tried for every head in this order; ``features``:
    per-input device features ``[N, D]`` (needed only by COSINE_TOPK
    candidates). Returns a dict with the configurations (baseline first), the
    mean errors ``E [C, H]``, the costs ``Omega [C, H]``, the chosen index per
    head and the resulting pattern table."""
    import torch

    if not calib:
        raise ValueError("at least one calibration input is needed")
    q0 = calib[0][0]
    H, N, _ = q0.shape
    configs = [(B.STRIDE, baseline_stride(sigma))] + [tuple(c) for c in candidates]
    C = len(configs)
    errors = np.zeros((C, H))
    costs = np.zeros((C, H))
    code = B._torch_dtype_code(q0)
    for n_in, (q, k, v) in enumerate(calib):
        full, _ = B.sparse_attention(q, k, v, [(B.DENSE, 0)] * H, frames, tokens_per_frame,
                                     stream=stream)
        for c, (pattern, param) in enumerate(configs):
            table = [(pattern, param)] * H
            idx = cnt = None
            if pattern == B.COSINE_TOPK:
                if features is None:
                    raise ValueError("COSINE_TOPK candidates need features")
                cap = B.index_capacity(table, frames, tokens_per_frame, code)
                nb = -(-N // B.BLOCK)
                idx = torch.empty((H, nb, cap), dtype=torch.int32, device=q.device)
                cnt = torch.empty((H, nb), dtype=torch.int32, device=q.device)
                B.cosine_select(features[n_in], table, frames, tokens_per_frame, idx, cnt,
                                stream=stream)
            elif pattern not in (B.DENSE, B.STRIDE):
                qp, kp = B.estimate_blocks(q, k, table, frames, tokens_per_frame, stream=stream)
                idx, cnt, _ = B.select_blocks(qp, kp, table, frames, tokens_per_frame, dtype=code,
                                              stream=stream)
            out, _ = B.sparse_attention(q, k, v, table, frames, tokens_per_frame, idx, cnt,
                                        stream=stream)
            errors[c] += B.nmse(full, out, frames, tokens_per_frame, stream=stream).cpu().numpy()
            if idx is None:
                costs[c] += attention_cost(pattern, param, N)
            else:
                ih, ch = idx.cpu().numpy(), cnt.cpu().numpy()
                costs[c] += [attention_cost(pattern, param, N, ih[h], ch[h]) for h in range(H)]
    errors /= len(calib)
    costs /= len(calib)
    choice = choose(errors, costs)
    return {"configs": configs, "errors": errors, "costs": costs, "choice": choice,
            "table": [configs[c] for c in choice]}


def choose(errors, costs) -> list:
    """Eq. 2 per head: ``errors``/``costs`` are ``[C, H]`` with row 0 the
    baseline. Walking the candidates in order, the choice moves to any
    candidate with a strictly lower error whose cost is not above the
    baseline's (ties keep the earlier entry)."""
    C, H = np.shape(errors)
    choice = []
    for h in range(H):
        best = 0
        for c in range(1, C):
            if costs[c][h] <= costs[0][h] and errors[c][h] < errors[best][h]:
                best = c
        choice.append(best)
    return choice

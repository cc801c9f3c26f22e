"""Seeded synthetic VGGT-shaped global-attention inputs.

Shapes follow the paper's feed-forward 3D reconstruction setting (Sec. 5.1):
518x518 images cut into 14x14 patches give 37x37 = 1369 patch tokens, plus
one camera and four register tokens per frame (1374 tokens), 16 heads of
width 64. Real image sequences and trained weights are not available, so the
values are synthetic, built to give the head behaviours of Sec. 3 (Obs. 2): a
per-frame shared low-rank component makes queries prefer keys of frames with
similar content, and large-norm keys on the five special tokens of every frame
give the vertical-line structure that query-probe Top-K heads target.

Recipe, per head h and frame f (all draws from one Philox stream per
(workload, seed, layer, head)):

* ``W[h,f]``: 4x64 with orthonormal rows (QR of a Gaussian 64x4);
* ``m[h,f] ~ N(0,1)^4`` per frame, ``C[h,f] ~ N(0,1)^(T x 4)`` per token;
* ``comp = 2 (m + C) W`` (the per-frame shared rank-4 component, scale 2);
* ``Q = Z_Q + comp``, ``K = Z_K + comp``, ``V = Z_V`` with ``Z ~ N(0,1)``;
* the K rows of the five special tokens of every frame are scaled by 4;
* values are rounded to bf16 (round to nearest even, bit arithmetic) or kept
  as fp32, and both consumers read the same bits.

The pattern table (one class and one Top-K budget per head) stands in for the
offline profiling output of Sec. 4.2, whose real tables are not published.
"""
from __future__ import annotations

import math
import os
import zlib
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from fractions import Fraction

import numpy as np

# Pattern classes; the integer codes are the C ABI's ``saf3r_pattern`` values.
DENSE = 0
FRAME_LOCAL = 1
TOPK = 2

HEADS = 16
HEAD_DIM = 64
BLOCK = 64
SPECIAL_TOKENS = 5  # 1 camera + 4 register tokens per frame
SPECIAL_KEY_SCALE = 4.0
COMPONENT_RANK = 4
COMPONENT_SCALE = 2.0
FRAME_LOCAL_HEADS = 6


@dataclass(frozen=True)
class Workload:
    """One global-attention workload: shapes, dtype and how its table is drawn.

    ``table_rule`` is one of
      * ``("fixed", n_dense, n_frame_local, topk_percent)``;
      * ``("sparsity", tau_percent)``: one common Top-K budget from a target
        overall block sparsity ``tau``;
      * ``("sparsity_pcts", tau_percent, pcts)``: per-head Top-K budgets drawn
        from ``pcts`` percent of the key blocks;
      * ``("sparsity_range", lo, hi)``: ``tau`` drawn per layer in [lo, hi].
    """

    name: str
    frames: int
    tokens_per_frame: int
    dtype: str  # "f32" or "bf16"
    table_rule: tuple
    layers: int = 1
    heads: int = HEADS
    head_dim: int = HEAD_DIM
    block: int = BLOCK
    description: str = field(default="", compare=False)

    @property
    def tokens(self) -> int:
        return self.frames * self.tokens_per_frame

    @property
    def nb(self) -> int:
        return num_blocks(self.tokens, self.block)


def num_blocks(n: int, block: int = BLOCK) -> int:
    return -(-n // block)


WORKLOADS = {
    w.name: w
    for w in [
        Workload(
            "S4xT261-f32", 4, 261, "f32", ("fixed", 4, 6, 10),
            description="4 frames x (5 special + 16x16 patches), fp32; 4 dense, "
                        "6 frame-local, 6 Top-K heads keeping 10% of key blocks",
        ),
        Workload(
            "S8xT1374-bf16", 8, 1374, "bf16", ("sparsity", 85),
            description="8 frames x (5 special + 37x37 patches), bf16, target "
                        "block sparsity 85%",
        ),
        Workload(
            "S32xT1374-bf16", 32, 1374, "bf16", ("sparsity_pcts", 92, (2, 5, 10, 20)),
            description="32 frames x 1374 tokens, bf16, target sparsity 92%, "
                        "per-head Top-K budgets from {2,5,10,20}% of key blocks",
        ),
        Workload(
            "S100xT1374-bf16", 100, 1374, "bf16", ("sparsity", 95),
            description="100 frames x 1374 tokens = 137400 tokens, bf16, target "
                        "block sparsity 95%",
        ),
        Workload(
            "S200xT1374-bf16-L24", 200, 1374, "bf16", ("sparsity_range", 80, 98), layers=24,
            description="24 layers of 200 frames x 1374 tokens = 274800 tokens, "
                        "bf16, per-layer sparsity drawn in [80%, 98%]",
        ),
    ]
}


def _workload_id(w: Workload) -> int:
    return zlib.crc32(w.name.encode()) & 0x7FFFFFFF


def _rng(w: Workload, seed: int, layer: int, head: int, stream: int) -> np.random.Generator:
    ss = np.random.SeedSequence([_workload_id(w), seed, layer, head, stream])
    return np.random.Generator(np.random.Philox(ss))


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bits.

    Inputs are finite by construction (no NaN handling)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = b >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += b
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _head_values(w: Workload, seed: int, layer: int, head: int):
    """fp32 Q, K, V of one head, each of shape [frames*T, D]."""
    S, T, D = w.frames, w.tokens_per_frame, w.head_dim
    r = COMPONENT_RANK
    g = _rng(w, seed, layer, head, 0)
    gauss = g.standard_normal((S, D, r))
    basis, _ = np.linalg.qr(gauss)  # [S, D, r], orthonormal columns
    m = g.standard_normal((S, 1, r))
    c = g.standard_normal((S, T, r))
    comp = np.matmul((COMPONENT_SCALE * (m + c)).astype(np.float32),
                     np.transpose(basis, (0, 2, 1)).astype(np.float32))  # [S, T, D]
    z = _rng(w, seed, layer, head, 1).standard_normal((3, S * T, D), dtype=np.float32)
    comp = comp.reshape(S * T, D)
    q, k, v = z[0], z[1], z[2]
    q += comp
    k += comp
    special = (np.arange(S * T) % T) < SPECIAL_TOKENS
    k[special] *= np.float32(SPECIAL_KEY_SCALE)
    return q, k, v


def make_qkv(w: Workload, layer: int = 0, seed: int = 0, heads=None):
    """Q, K, V as ``[H, N, D]`` arrays.

    bf16 workloads return uint16 bf16 bit patterns, fp32 workloads float32."""
    heads = range(w.heads) if heads is None else heads
    H, N, D = len(heads), w.tokens, w.head_dim
    out_dtype = np.uint16 if w.dtype == "bf16" else np.float32
    q = np.empty((H, N, D), out_dtype)
    k = np.empty((H, N, D), out_dtype)
    v = np.empty((H, N, D), out_dtype)

    def fill(hi_h):
        hi, h = hi_h
        hq, hk, hv = _head_values(w, seed, layer, h)
        if w.dtype == "bf16":
            q[hi], k[hi], v[hi] = bf16_bits_from_f32(hq), bf16_bits_from_f32(hk), bf16_bits_from_f32(hv)
        else:
            q[hi], k[hi], v[hi] = hq, hk, hv

    # Heads are independent streams; numpy releases the GIL in the bulk work.
    workers = max(1, min(len(heads), 8, os.cpu_count() or 1))
    with ThreadPoolExecutor(workers) as pool:
        list(pool.map(fill, enumerate(heads)))
    return q, k, v


def _ceil_frac(x: Fraction) -> int:
    return -((-x.numerator) // x.denominator)


def layer_tau(w: Workload, layer: int, seed: int = 0) -> int:
    """Target overall block sparsity of a layer, in percent."""
    rule = w.table_rule
    if rule[0] in ("sparsity", "sparsity_pcts"):
        return rule[1]
    if rule[0] == "sparsity_range":
        g = _rng(w, seed, layer, 0x7FFFFFF1, 2)
        return int(g.integers(rule[1], rule[2] + 1))
    return -1


def make_table(w: Workload, layer: int = 0, seed: int = 0):
    """Per-head ``(pattern, topk_blocks)`` pairs; classes assigned by a seeded
    permutation of the heads.

    The Top-K budget is set so that the table's overall kept-block fraction is
    roughly ``1 - tau``, counting a frame-local head as keeping about ``1/S``
    of the key blocks; the achieved sparsity is measured, not assumed."""
    H, nb, S = w.heads, w.nb, w.frames
    rule = w.table_rule
    g = _rng(w, seed, layer, 0x7FFFFFF0, 3)
    if rule[0] == "fixed":
        n_dense, n_fl, pct = rule[1], rule[2], rule[3]
        n_topk = H - n_dense - n_fl
        ks = [max(1, min(nb, _ceil_frac(Fraction(pct * nb, 100))))] * n_topk
    else:
        tau = layer_tau(w, layer, seed)
        n_dense = (H * (100 - tau)) // 200
        n_fl = FRAME_LOCAL_HEADS
        n_topk = H - n_dense - n_fl
        if rule[0] == "sparsity_pcts":
            pcts = g.choice(np.asarray(rule[2]), size=n_topk)
            ks = [max(1, min(nb, _ceil_frac(Fraction(int(p) * nb, 100)))) for p in pcts]
        else:
            budget = Fraction(H * (100 - tau), 100) - n_dense - Fraction(n_fl, S)
            rho = budget / n_topk
            k = max(1, min(nb, _ceil_frac(rho * nb)))
            ks = [k] * n_topk
    classes = [DENSE] * n_dense + [FRAME_LOCAL] * n_fl + [TOPK] * n_topk
    topks = [0] * n_dense + [0] * n_fl + ks
    perm = g.permutation(H)
    table = [None] * H
    for slot, h in enumerate(perm):
        table[int(h)] = (classes[slot], int(topks[slot]))
    return table


def make_layer(w: Workload, layer: int = 0, seed: int = 0):
    q, k, v = make_qkv(w, layer, seed)
    return q, k, v, make_table(w, layer, seed)


def dense_table(w: Workload):
    return [(DENSE, 0)] * w.heads


def _self_check():
    w = WORKLOADS["S8xT1374-bf16"]
    assert w.nb == 172 and math.isclose(w.tokens / 64, 171.75)


_self_check()

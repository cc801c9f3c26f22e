"""Python binding of libsaf3r.so (ctypes): argument marshalling only.

Every computation runs in the HIP library; PyTorch only provides device
memory and the current HIP stream. Names mirror the C ABI without the
``saf3r_`` prefix. If the library has not been built, ``load()`` raises.
The library is ``libsaf3r.so`` next to this file, or the file the
environment variable ``SAF3R_LIBRARY`` names.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("SAF3R_LIBRARY") or os.path.join(PKG, "libsaf3r.so")

F32, BF16 = 0, 1
DENSE, FRAME_LOCAL, TOPK, ANCHOR, STRIDE, GLOBAL_PROBE, COSINE_TOPK, SKIP = 0, 1, 2, 3, 4, 5, 6, 7
HEAD_DIM = 64
BLOCK = 64

EXPORTS = (
    "saf3r_num_blocks",
    "saf3r_index_capacity",
    "saf3r_estimate_blocks",
    "saf3r_select_blocks",
    "saf3r_select_workspace_bytes",
    "saf3r_sparse_attention",
    "saf3r_attention_workspace_bytes",
    "saf3r_cosine_workspace_bytes",
    "saf3r_cosine_select",
    "saf3r_nmse_workspace_bytes",
    "saf3r_nmse",
    "saf3r_nmse_noalloc",
    "saf3r_validate_index",
    "saf3r_status_string",
)

CORRUPT_INDEX = -6  # saf3r_validate_index: a list breaks its form


class Problem(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("heads", "frames", "tokens_per_frame", "head_dim", "block", "dtype")]


class HeadCfg(ctypes.Structure):
    _fields_ = [("pattern", ctypes.c_int32), ("param", ctypes.c_int32)]


class Saf3rError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        msg = _lib().saf3r_status_string(status).decode() if _LIB else str(status)
        super().__init__(f"{where}: status {status} ({msg})")


_LIB = None


def _declare(lib):
    P, C, V, I32 = ctypes.POINTER(Problem), ctypes.POINTER(HeadCfg), ctypes.c_void_p, ctypes.c_int32
    lib.saf3r_num_blocks.argtypes = [P]
    lib.saf3r_num_blocks.restype = I32
    lib.saf3r_index_capacity.argtypes = [P, C]
    lib.saf3r_index_capacity.restype = I32
    lib.saf3r_estimate_blocks.argtypes = [P, C, V, V, V, V, V]
    lib.saf3r_estimate_blocks.restype = I32
    lib.saf3r_select_blocks.argtypes = [P, C, V, V, V, V, I32, V, V, ctypes.c_int64, V]
    lib.saf3r_select_blocks.restype = I32
    lib.saf3r_select_workspace_bytes.argtypes = [P, C]
    lib.saf3r_select_workspace_bytes.restype = ctypes.c_int64
    lib.saf3r_sparse_attention.argtypes = [P, C, V, V, V, V, V, I32, V, V, V, ctypes.c_int64, V]
    lib.saf3r_sparse_attention.restype = I32
    lib.saf3r_attention_workspace_bytes.argtypes = [P, C]
    lib.saf3r_attention_workspace_bytes.restype = ctypes.c_int64
    lib.saf3r_cosine_workspace_bytes.argtypes = [P, I32]
    lib.saf3r_cosine_workspace_bytes.restype = ctypes.c_int64
    lib.saf3r_cosine_select.argtypes = [P, C, V, I32, V, ctypes.c_int64, V, V, I32, V]
    lib.saf3r_cosine_select.restype = I32
    lib.saf3r_nmse_workspace_bytes.argtypes = [P]
    lib.saf3r_nmse_workspace_bytes.restype = ctypes.c_int64
    lib.saf3r_nmse.argtypes = [P, V, V, V, ctypes.c_int64, V, V]
    lib.saf3r_nmse.restype = I32
    lib.saf3r_nmse_noalloc.argtypes = [P, V, V, V, V]
    lib.saf3r_nmse_noalloc.restype = I32
    lib.saf3r_validate_index.argtypes = [P, C, V, V, I32, V, ctypes.POINTER(I32), V]
    lib.saf3r_validate_index.restype = I32
    lib.saf3r_status_string.argtypes = [I32]
    lib.saf3r_status_string.restype = ctypes.c_char_p


def load(path: str = None):
    """Load the HIP library (raises if it has not been built)."""
    global _LIB
    path = path or LIB_PATH
    if _LIB is None:
        if not os.path.exists(path):
            raise RuntimeError(
                f"{path} is missing: build it with `python -m paper_2607_03612_amd.build`")
        lib = ctypes.CDLL(path)
        _declare(lib)
        _LIB = lib
    return _LIB


def _lib():
    return load()


# ------------------------------------------------------------ marshalling


def problem(heads: int, frames: int, tokens_per_frame: int, dtype: int) -> Problem:
    return Problem(heads, frames, tokens_per_frame, HEAD_DIM, BLOCK, dtype)


def head_table(table) -> ctypes.Array:
    """Per-head ``(pattern, param)`` pairs as the C array."""
    arr = (HeadCfg * len(table))()
    for h, (pattern, param) in enumerate(table):
        arr[h] = HeadCfg(int(pattern), int(param))
    return arr


def _torch_dtype_code(t) -> int:
    import torch

    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise ValueError(f"unsupported dtype {t.dtype}")


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(status: int, where: str):
    if status != 0:
        raise Saf3rError(status, where)


def _check_qkv(*ts):
    t0 = ts[0]
    for t in ts:
        if not (t.is_cuda and t.is_contiguous() and t.dim() == 3 and t.shape[2] == HEAD_DIM):
            raise ValueError("expected contiguous device tensors of shape [heads, N, 64]")
        if t.shape != t0.shape or t.dtype != t0.dtype or t.device != t0.device:
            raise ValueError("q, k, v must share shape, dtype and device")


def num_blocks(heads, frames, tokens_per_frame, dtype=BF16) -> int:
    p = problem(heads, frames, tokens_per_frame, dtype)
    r = _lib().saf3r_num_blocks(ctypes.byref(p))
    _check(min(r, 0), "saf3r_num_blocks")
    return r


def index_capacity(table, frames, tokens_per_frame, dtype=BF16) -> int:
    p = problem(len(table), frames, tokens_per_frame, dtype)
    r = _lib().saf3r_index_capacity(ctypes.byref(p), head_table(table))
    _check(min(r, 0), "saf3r_index_capacity")
    return r


def estimate_blocks(q, k, table, frames, tokens_per_frame, q_pooled=None, k_pooled=None,
                    stream=None):
    """Pooled Q ``[heads, nb, 64]`` and pooled K ``[heads, 64, nb]`` (float64;
    TOPK and GLOBAL_PROBE heads only)."""
    import torch

    _check_qkv(q, k)
    H, N, _ = q.shape
    if frames * tokens_per_frame != N or len(table) != H:
        raise ValueError("frames * tokens_per_frame must equal N and len(table) the heads")
    nb = -(-N // BLOCK)
    if q_pooled is None:
        q_pooled = torch.zeros((H, nb, HEAD_DIM), dtype=torch.float64, device=q.device)
    if k_pooled is None:
        k_pooled = torch.zeros((H, HEAD_DIM, nb), dtype=torch.float64, device=q.device)
    p = problem(H, frames, tokens_per_frame, _torch_dtype_code(q))
    _check(_lib().saf3r_estimate_blocks(ctypes.byref(p), head_table(table), _ptr(q), _ptr(k),
                                        _ptr(q_pooled), _ptr(k_pooled), _stream(stream)),
           "saf3r_estimate_blocks")
    return q_pooled, k_pooled


def select_workspace_bytes(table, frames, tokens_per_frame, dtype=BF16) -> int:
    """Bytes of the workspace that lets saf3r_select_blocks take every TOPK
    head in one batch (0 without TOPK heads)."""
    p = problem(len(table), frames, tokens_per_frame, dtype)
    r = _lib().saf3r_select_workspace_bytes(ctypes.byref(p), head_table(table))
    _check(min(r, 0), "saf3r_select_workspace_bytes")
    return int(r)


def select_blocks(q_pooled, k_pooled, table, frames, tokens_per_frame, cap=None,
                  block_idx=None, block_cnt=None, want_scores=False, dtype=BF16, workspace=None,
                  stream=None):
    """Kept key-block lists: ``(block_idx [H, nb, cap], block_cnt [H, nb], scores or None)``.

    ``workspace``: None for the single-launch path, or a contiguous device
    tensor (any dtype, 16-byte aligned) for the two-launch path; see
    ``select_workspace_bytes``."""
    import torch

    H, nb, _ = q_pooled.shape
    for t, shape in ((q_pooled, (H, nb, HEAD_DIM)), (k_pooled, (H, HEAD_DIM, nb))):
        if not (t.is_cuda and t.is_contiguous() and t.dtype == torch.float64 and t.shape == shape):
            raise ValueError("pooled tensors must be contiguous float64 device tensors, "
                             "q [heads, nb, 64] and k [heads, 64, nb]")
    if cap is None:
        cap = index_capacity(table, frames, tokens_per_frame, dtype)
    dev = q_pooled.device
    if block_idx is None:
        block_idx = torch.empty((H, nb, cap), dtype=torch.int32, device=dev)
    if block_cnt is None:
        block_cnt = torch.empty((H, nb), dtype=torch.int32, device=dev)
    scores = torch.zeros((H, nb, nb), dtype=torch.float64, device=dev) if want_scores else None
    p = problem(H, frames, tokens_per_frame, dtype)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib().saf3r_select_blocks(ctypes.byref(p), head_table(table), _ptr(q_pooled),
                                      _ptr(k_pooled), _ptr(block_idx), _ptr(block_cnt), int(cap),
                                      _ptr(scores), _ptr(workspace), ctypes.c_int64(ws_bytes),
                                      _stream(stream)),
           "saf3r_select_blocks")
    return block_idx, block_cnt, scores


def attention_workspace_bytes(table, frames, tokens_per_frame, dtype=BF16) -> int:
    """Bytes of the workspace that lets saf3r_sparse_attention split its long
    lists into key ranges (0 if no head qualifies)."""
    p = problem(len(table), frames, tokens_per_frame, dtype)
    r = _lib().saf3r_attention_workspace_bytes(ctypes.byref(p), head_table(table))
    _check(min(r, 0), "saf3r_attention_workspace_bytes")
    return int(r)


def sparse_attention(q, k, v, table, frames, tokens_per_frame, block_idx=None, block_cnt=None,
                     out=None, want_lse=False, workspace=None, stream=None):
    """Attention over the kept keys: ``(out [H, N, 64], lse [H, N] float32 or None)``.

    ``workspace``: None, or a contiguous device tensor (any dtype, 16-byte
    aligned) of at least ``attention_workspace_bytes`` bytes, with which long
    lists run split into key ranges."""
    import torch

    _check_qkv(q, k, v)
    H, N, _ = q.shape
    if frames * tokens_per_frame != N or len(table) != H:
        raise ValueError("frames * tokens_per_frame must equal N and len(table) the heads")
    cap = 0 if block_idx is None else int(block_idx.shape[2])
    if out is None:
        out = torch.empty_like(q)
    lse = torch.empty((H, N), dtype=torch.float32, device=q.device) if want_lse else None
    p = problem(H, frames, tokens_per_frame, _torch_dtype_code(q))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib().saf3r_sparse_attention(ctypes.byref(p), head_table(table), _ptr(q), _ptr(k),
                                         _ptr(v), _ptr(block_idx), _ptr(block_cnt), cap, _ptr(out),
                                         _ptr(lse), _ptr(workspace), ctypes.c_int64(ws_bytes),
                                         _stream(stream)),
           "saf3r_sparse_attention")
    return out, lse


def cosine_workspace_bytes(frames, tokens_per_frame, feat_dim, heads=1, dtype=BF16) -> int:
    p = problem(heads, frames, tokens_per_frame, dtype)
    r = _lib().saf3r_cosine_workspace_bytes(ctypes.byref(p), int(feat_dim))
    _check(min(r, 0), "saf3r_cosine_workspace_bytes")
    return int(r)


def cosine_select(features, table, frames, tokens_per_frame, block_idx, block_cnt, workspace=None,
                  stream=None):
    """Per-frame cosine Top-K lists of the COSINE_TOPK heads, written into
    ``block_idx [H, nb, cap]`` / ``block_cnt [H, nb]`` (other heads' rows
    untouched). ``features``: device ``[N, feat_dim]`` of the layer dtype."""
    import torch

    if not (features.is_cuda and features.is_contiguous() and features.dim() == 2):
        raise ValueError("features must be a contiguous device tensor [N, feat_dim]")
    N, D = features.shape
    if frames * tokens_per_frame != N:
        raise ValueError("frames * tokens_per_frame must equal the feature rows")
    code = _torch_dtype_code(features)
    H = len(table)
    nbytes = cosine_workspace_bytes(frames, tokens_per_frame, D, H, code)
    if workspace is None:
        workspace = torch.empty(nbytes // 8, dtype=torch.float64, device=features.device)
    p = problem(H, frames, tokens_per_frame, code)
    _check(_lib().saf3r_cosine_select(ctypes.byref(p), head_table(table), _ptr(features), int(D),
                                      _ptr(workspace), int(workspace.numel() * workspace.element_size()),
                                      _ptr(block_idx), _ptr(block_cnt), int(block_idx.shape[2]),
                                      _stream(stream)),
           "saf3r_cosine_select")
    return block_idx, block_cnt


def nmse_workspace_bytes(heads, frames, tokens_per_frame, dtype=BF16) -> int:
    p = problem(heads, frames, tokens_per_frame, dtype)
    r = _lib().saf3r_nmse_workspace_bytes(ctypes.byref(p))
    _check(min(r, 0), "saf3r_nmse_workspace_bytes")
    return int(r)


def nmse(o_full, o_sparse, frames, tokens_per_frame, out=None, workspace=None, stream=None):
    """Per-head ``||o_full - o_sparse||^2 / ||o_full||^2`` (float64 ``[H]``)."""
    import torch

    _check_qkv(o_full, o_sparse)
    H, N, _ = o_full.shape
    dtype = _torch_dtype_code(o_full)
    if out is None:
        out = torch.empty(H, dtype=torch.float64, device=o_full.device)
    need = nmse_workspace_bytes(H, frames, tokens_per_frame, dtype)
    if workspace is None:
        workspace = torch.empty(need // 8, dtype=torch.float64, device=o_full.device)
    p = problem(H, frames, tokens_per_frame, dtype)
    _check(_lib().saf3r_nmse(ctypes.byref(p), _ptr(o_full), _ptr(o_sparse), _ptr(workspace),
                             ctypes.c_int64(workspace.numel() * workspace.element_size()),
                             _ptr(out), _stream(stream)), "saf3r_nmse")
    return out


def nmse_noalloc(o_full, o_sparse, frames, tokens_per_frame, out, stream=None):
    """``nmse`` through the entry point that allocates nothing: the library's
    own per-GPU array holds the partial sums. ``out``: float64 ``[H]`` device
    tensor the caller provides."""
    _check_qkv(o_full, o_sparse)
    H, N, _ = o_full.shape
    p = problem(H, frames, tokens_per_frame, _torch_dtype_code(o_full))
    _check(_lib().saf3r_nmse_noalloc(ctypes.byref(p), _ptr(o_full), _ptr(o_sparse), _ptr(out),
                                     _stream(stream)), "saf3r_nmse_noalloc")
    return out


def validate_index(block_idx, block_cnt, table, frames, tokens_per_frame, workspace=None,
                   dtype=BF16, stream=None):
    """Checks the kept-block lists of the listed heads (count, strictly
    ascending entries in range, -1 padding); waits for the stream. Returns
    ``None`` when every row passes, else the lowest failing row as
    ``(head, query_block)``."""
    import torch

    H, nb, cap = block_idx.shape
    if block_cnt.shape != (H, nb) or len(table) != H:
        raise ValueError("block_idx [H, nb, cap], block_cnt [H, nb] and the table must agree")
    if workspace is None:
        workspace = torch.empty(2, dtype=torch.int32, device=block_idx.device)
    p = problem(H, frames, tokens_per_frame, dtype)
    first = ctypes.c_int32(-1)
    st = _lib().saf3r_validate_index(ctypes.byref(p), head_table(table), _ptr(block_idx),
                                     _ptr(block_cnt), ctypes.c_int32(cap), _ptr(workspace),
                                     ctypes.byref(first), _stream(stream))
    if st == CORRUPT_INDEX:
        return divmod(first.value, nb)
    _check(st, "saf3r_validate_index")
    return None


def run_layer(q, k, v, table, frames, tokens_per_frame, stream=None):
    """estimate -> select -> attend for one layer; returns (out, block_idx, block_cnt)."""
    dtype = _torch_dtype_code(q)
    qp, kp = estimate_blocks(q, k, table, frames, tokens_per_frame, stream=stream)
    idx, cnt, _ = select_blocks(qp, kp, table, frames, tokens_per_frame, dtype=dtype, stream=stream)
    out, _ = sparse_attention(q, k, v, table, frames, tokens_per_frame, idx, cnt, stream=stream)
    return out, idx, cnt

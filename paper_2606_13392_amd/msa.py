"""Python binding of libmsa.so (argument marshalling only).

Each function checks dtypes, shapes and devices, takes device pointers and the
current torch stream, and calls the C ABI of ``include/msa.h`` under the same
name.  All work runs in the library's HIP kernels; there is no fallback: when
the library is not built, or a call returns an error, a RuntimeError is raised.
torch provides device memory (outputs, workspaces) and the stream.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmsa.so")

MSA_OK, MSA_ERR_INVALID, MSA_ERR_UNSUPPORTED, MSA_ERR_WORKSPACE, MSA_ERR_HIP = 0, -1, -2, -3, -4

EXPORTS = [
    "msa_strerror",
    "msa_index_topk_workspace_size", "msa_index_topk", "msa_index_topk_noalloc", "msa_block_topk",
    "msa_sparse_attn_prefill_workspace_size", "msa_sparse_attn_prefill",
    "msa_sparse_attn_decode_workspace_size", "msa_sparse_attn_decode",
    "msa_sparse_attn_prefill_fp8", "msa_sparse_attn_decode_fp8",
    "msa_dense_attn_workspace_size", "msa_dense_attn",
    "msa_sparse_attn_backward_workspace_size", "msa_sparse_attn_backward",
    "msa_sparse_kl_backward_workspace_size", "msa_sparse_kl_backward",
    "msa_profile_enable", "msa_profile_reset", "msa_profile_kernel_name", "msa_profile_read",
]


class MsaSeqsC(ctypes.Structure):
    _fields_ = [
        ("num_seqs", ctypes.c_int32),
        ("total_q_rows", ctypes.c_int64),
        ("total_kv_rows", ctypes.c_int64),
        ("max_q_rows", ctypes.c_int32),
        ("max_kv_len", ctypes.c_int32),
        ("q_offsets", ctypes.c_void_p),
        ("kv_starts", ctypes.c_void_p),
        ("kv_lens", ctypes.c_void_p),
        ("block_table", ctypes.c_void_p),
        ("block_table_stride", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libmsa.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, S, I, Z, F = ctypes.c_void_p, ctypes.POINTER(MsaSeqsC), ctypes.c_int, ctypes.c_size_t, ctypes.c_float
        L.msa_strerror.argtypes = [I]
        L.msa_strerror.restype = ctypes.c_char_p
        L.msa_index_topk_workspace_size.argtypes = [S, I, I, I, I]
        L.msa_index_topk_workspace_size.restype = Z
        L.msa_index_topk.argtypes = [P, P, S, I, I, I, I, P, P, Z, P]
        L.msa_index_topk.restype = I
        L.msa_index_topk_noalloc.argtypes = [P, P, S, I, I, I, I, P, P]
        L.msa_index_topk_noalloc.restype = I
        L.msa_block_topk.argtypes = [P, ctypes.c_int64, I, ctypes.c_int64, I, P, P]
        L.msa_block_topk.restype = I
        for name in ("prefill", "decode"):
            ws = getattr(L, f"msa_sparse_attn_{name}_workspace_size")
            ws.argtypes = [S, I, I, I, I, I]
            ws.restype = Z
            fn = getattr(L, f"msa_sparse_attn_{name}")
            fn.argtypes = [P, P, P, P, S, I, I, I, I, I, F, P, P, P, Z, P]
            fn.restype = I
        for name in ("prefill", "decode"):
            fn = getattr(L, f"msa_sparse_attn_{name}_fp8")
            fn.argtypes = [P, P, P, F, F, F, P, S, I, I, I, I, I, F, P, P, P, Z, P]
            fn.restype = I
        L.msa_dense_attn_workspace_size.argtypes = [S, I, I, I]
        L.msa_dense_attn_workspace_size.restype = Z
        L.msa_dense_attn.argtypes = [P, P, P, S, I, I, I, F, P, P, P, Z, P]
        L.msa_dense_attn.restype = I
        L.msa_sparse_attn_backward_workspace_size.argtypes = [S, I, I, I, I, I]
        L.msa_sparse_attn_backward_workspace_size.restype = Z
        L.msa_sparse_attn_backward.argtypes = [P, P, P, P, P, P, P, S, I, I, I, I, I, F, P, P, P, P, Z, P]
        L.msa_sparse_attn_backward.restype = I
        L.msa_sparse_kl_backward_workspace_size.argtypes = [S, I, I, I, I, I, I]
        L.msa_sparse_kl_backward_workspace_size.restype = Z
        L.msa_sparse_kl_backward.argtypes = [P, P, P, P, P, P, S, I, I, I, I, I, I, F, F, P, P, P, P, Z, P]
        L.msa_sparse_kl_backward.restype = I
        L.msa_profile_enable.argtypes = [I]
        L.msa_profile_enable.restype = I
        L.msa_profile_reset.argtypes = []
        L.msa_profile_reset.restype = I
        L.msa_profile_kernel_name.argtypes = [I]
        L.msa_profile_kernel_name.restype = ctypes.c_char_p
        L.msa_profile_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_int64),
                                       ctypes.POINTER(ctypes.c_double)]
        L.msa_profile_read.restype = I
        _lib = L
    return _lib


def _check(status: int, what: str):
    if status != MSA_OK:
        raise RuntimeError(f"{what} failed: {lib().msa_strerror(status).decode()} ({status})")


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _need(t: torch.Tensor, name: str, dtype: torch.dtype, shape: Sequence[int], device):
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if t.device != device:
        raise ValueError(f"{name}: expected device {device}, got {t.device}")


class Seqs:
    """Sequence layout (see include/msa.h): device arrays plus host totals.

    ``block_table`` (int32 [num_seqs, max_blocks] on the device) makes the key
    side paged with pages of ``page_size`` rows; ``kv_starts`` is then unused."""

    def __init__(self, q_rows: Sequence[int], kv_lens: Sequence[int], kv_starts: Sequence[int],
                 total_kv_rows: int, device, block_table: Optional[torch.Tensor] = None, page_size: int = 0):
        assert len(q_rows) == len(kv_lens) == len(kv_starts) and len(q_rows) >= 1
        offs = [0]
        for r in q_rows:
            offs.append(offs[-1] + int(r))
        dev = torch.device(device)
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        self.q_offsets = torch.tensor(offs, dtype=torch.int32, device=self.device)
        self.kv_starts = torch.tensor([int(x) for x in kv_starts], dtype=torch.int64, device=self.device)
        self.kv_lens = torch.tensor([int(x) for x in kv_lens], dtype=torch.int32, device=self.device)
        self.num_seqs = len(q_rows)
        self.total_q_rows = offs[-1]
        self.total_kv_rows = int(total_kv_rows)
        self.max_q_rows = max(int(r) for r in q_rows)
        self.max_kv_len = max(int(x) for x in kv_lens)
        self.block_table = block_table
        if block_table is not None:
            _need(block_table, "block_table", torch.int32, (self.num_seqs, block_table.shape[1]), self.device)
        self.c = MsaSeqsC(self.num_seqs, self.total_q_rows, self.total_kv_rows, self.max_q_rows,
                          self.max_kv_len, self.q_offsets.data_ptr(), self.kv_starts.data_ptr(),
                          self.kv_lens.data_ptr(), None if block_table is None else block_table.data_ptr(),
                          0 if block_table is None else int(block_table.shape[1]), int(page_size))

    @classmethod
    def from_problem(cls, p, device) -> "Seqs":
        return cls(p.q_rows, p.kv_lens, p.kv_starts, p.total_kv_rows, device)

    def ref(self):
        return ctypes.byref(self.c)


def _workspace(nbytes: int, device, ws: Optional[torch.Tensor]) -> Optional[torch.Tensor]:
    """The caller's workspace as given (a call runs in chunks sized to it and
    reports MSA_ERR_WORKSPACE below its minimum), else one of the queried size."""
    if ws is not None or nbytes == 0:
        return ws
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


# ---------------------------------------------------------------- Index Branch
def index_topk_workspace_size(seqs: Seqs, num_kv_heads: int, d_idx: int, block_size: int, topk: int) -> int:
    return int(lib().msa_index_topk_workspace_size(seqs.ref(), num_kv_heads, d_idx, block_size, topk))


def index_topk(index_q: torch.Tensor, index_k: torch.Tensor, seqs: Seqs, block_size: int, topk: int,
               out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Block ids [total_q_rows, H_kv, topk] (int32, ascending, -1 padded)."""
    Tq, H_kv, d_idx = index_q.shape
    dev = seqs.device
    _need(index_q, "index_q", torch.bfloat16, (seqs.total_q_rows, H_kv, d_idx), dev)
    _need(index_k, "index_k", torch.bfloat16, (seqs.total_kv_rows, d_idx), dev)
    if out is None:
        out = torch.empty((Tq, H_kv, topk), dtype=torch.int32, device=dev)
    _need(out, "block_ids", torch.int32, (Tq, H_kv, topk), dev)
    nbytes = index_topk_workspace_size(seqs, H_kv, d_idx, block_size, topk)
    ws = _workspace(nbytes, dev, workspace)
    st = lib().msa_index_topk(_ptr(index_q), _ptr(index_k), seqs.ref(), H_kv, d_idx, block_size, topk,
                              _ptr(out), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(), _stream())
    _check(st, "msa_index_topk")
    return out


NOALLOC_MAX_BYTES = 64 << 20      # MSA_INDEX_TOPK_NOALLOC_MAX_BYTES


def index_topk_noalloc(index_q: torch.Tensor, index_k: torch.Tensor, seqs: Seqs, block_size: int, topk: int,
                       out: torch.Tensor) -> torch.Tensor:
    """msa_index_topk_noalloc: the Index Branch on the library's own scratch
    array; ``out`` (int32 [total_q_rows, H_kv, topk]) is caller-allocated."""
    Tq, H_kv, d_idx = index_q.shape
    dev = seqs.device
    _need(index_q, "index_q", torch.bfloat16, (seqs.total_q_rows, H_kv, d_idx), dev)
    _need(index_k, "index_k", torch.bfloat16, (seqs.total_kv_rows, d_idx), dev)
    _need(out, "block_ids", torch.int32, (Tq, H_kv, topk), dev)
    st = lib().msa_index_topk_noalloc(_ptr(index_q), _ptr(index_k), seqs.ref(), H_kv, d_idx, block_size, topk,
                                      _ptr(out), _stream())
    _check(st, "msa_index_topk_noalloc")
    return out


def block_topk(scores: torch.Tensor, k: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """msa_block_topk: the k best columns of each row of an fp32 [n_rows, n_cols]
    matrix (row stride taken from the tensor; unit column stride), int32
    [n_rows, k], ascending, -1 padded."""
    if scores.dim() != 2:
        raise ValueError("scores: expected a 2-d tensor")
    if scores.dtype != torch.float32:
        raise TypeError(f"scores: expected torch.float32, got {scores.dtype}")
    n_rows, n_cols = scores.shape
    if n_cols > 1 and scores.stride(1) != 1:
        raise ValueError("scores: columns must be contiguous")
    ld = scores.stride(0) if n_rows > 1 else max(n_cols, 1)
    dev = scores.device
    if out is None:
        out = torch.empty((n_rows, k), dtype=torch.int32, device=dev)
    _need(out, "ids", torch.int32, (n_rows, k), dev)
    st = lib().msa_block_topk(_ptr(scores), n_rows, n_cols, ld, k, _ptr(out), _stream())
    _check(st, "msa_block_topk")
    return out


# ---------------------------------------------------------------- Main Branch
def _attn(kind: str, q, k, v, block_ids, seqs: Seqs, block_size: int, softmax_scale, out, lse, workspace):
    Tq, H_q, d_h = q.shape
    H_kv = k.shape[1]
    topk = block_ids.shape[2]
    dev = seqs.device
    _need(q, "q", torch.bfloat16, (seqs.total_q_rows, H_q, d_h), dev)
    _need(k, "k", torch.bfloat16, (seqs.total_kv_rows, H_kv, d_h), dev)
    _need(v, "v", torch.bfloat16, (seqs.total_kv_rows, H_kv, d_h), dev)
    _need(block_ids, "block_ids", torch.int32, (Tq, H_kv, topk), dev)
    if out is None:
        out = torch.empty((Tq, H_q, d_h), dtype=torch.bfloat16, device=dev)
    if lse is None:
        lse = torch.empty((Tq, H_q), dtype=torch.float32, device=dev)
    _need(out, "o", torch.bfloat16, (Tq, H_q, d_h), dev)
    _need(lse, "lse", torch.float32, (Tq, H_q), dev)
    scale = 1.0 / math.sqrt(d_h) if softmax_scale is None else float(softmax_scale)
    L = lib()
    nbytes = int(getattr(L, f"msa_sparse_attn_{kind}_workspace_size")(seqs.ref(), H_q, H_kv, d_h, block_size, topk))
    ws = _workspace(nbytes, dev, workspace)
    st = getattr(L, f"msa_sparse_attn_{kind}")(
        _ptr(q), _ptr(k), _ptr(v), _ptr(block_ids), seqs.ref(), H_q, H_kv, d_h, block_size, topk, scale,
        _ptr(out), _ptr(lse), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(), _stream())
    _check(st, f"msa_sparse_attn_{kind}")
    return out, lse


def sparse_attn_prefill_workspace_size(seqs: Seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk) -> int:
    return int(lib().msa_sparse_attn_prefill_workspace_size(seqs.ref(), num_q_heads, num_kv_heads, head_dim,
                                                             block_size, topk))


def sparse_attn_decode_workspace_size(seqs: Seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk) -> int:
    return int(lib().msa_sparse_attn_decode_workspace_size(seqs.ref(), num_q_heads, num_kv_heads, head_dim,
                                                            block_size, topk))


def sparse_attn_prefill(q, k, v, block_ids, seqs: Seqs, block_size: int, softmax_scale=None,
                        out=None, lse=None, workspace=None):
    """O [Tq, H_q, d_h] bf16 and LSE [Tq, H_q] fp32 over the selected blocks."""
    return _attn("prefill", q, k, v, block_ids, seqs, block_size, softmax_scale, out, lse, workspace)


def sparse_attn_decode(q, k, v, block_ids, seqs: Seqs, block_size: int, softmax_scale=None,
                       out=None, lse=None, workspace=None):
    """Decode-shaped variant of sparse_attn_prefill (one query row per sequence)."""
    return _attn("decode", q, k, v, block_ids, seqs, block_size, softmax_scale, out, lse, workspace)


def _attn_fp8(kind: str, q, k, v, scales, block_ids, seqs: Seqs, block_size: int, softmax_scale, out, lse,
              workspace):
    Tq, H_q, d_h = q.shape
    H_kv = k.shape[1]
    topk = block_ids.shape[2]
    dev = seqs.device
    _need(q, "q", torch.uint8, (seqs.total_q_rows, H_q, d_h), dev)
    _need(k, "k", torch.uint8, (seqs.total_kv_rows, H_kv, d_h), dev)
    _need(v, "v", torch.uint8, (seqs.total_kv_rows, H_kv, d_h), dev)
    _need(block_ids, "block_ids", torch.int32, (Tq, H_kv, topk), dev)
    if out is None:
        out = torch.empty((Tq, H_q, d_h), dtype=torch.bfloat16, device=dev)
    if lse is None:
        lse = torch.empty((Tq, H_q), dtype=torch.float32, device=dev)
    _need(out, "o", torch.bfloat16, (Tq, H_q, d_h), dev)
    _need(lse, "lse", torch.float32, (Tq, H_q), dev)
    scale = 1.0 / math.sqrt(d_h) if softmax_scale is None else float(softmax_scale)
    L = lib()
    nbytes = int(getattr(L, f"msa_sparse_attn_{kind}_workspace_size")(seqs.ref(), H_q, H_kv, d_h, block_size, topk))
    ws = _workspace(nbytes, dev, workspace)
    qs, ks, vs = (float(x) for x in scales)
    st = getattr(L, f"msa_sparse_attn_{kind}_fp8")(
        _ptr(q), _ptr(k), _ptr(v), qs, ks, vs, _ptr(block_ids), seqs.ref(), H_q, H_kv, d_h, block_size, topk, scale,
        _ptr(out), _ptr(lse), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(), _stream())
    _check(st, f"msa_sparse_attn_{kind}_fp8")
    return out, lse


def sparse_attn_prefill_fp8(q, k, v, scales, block_ids, seqs: Seqs, block_size: int, softmax_scale=None,
                            out=None, lse=None, workspace=None):
    """Main Branch on e4m3 codes (uint8 tensors) with per-tensor scales (q, k, v)."""
    return _attn_fp8("prefill", q, k, v, scales, block_ids, seqs, block_size, softmax_scale, out, lse, workspace)


def sparse_attn_decode_fp8(q, k, v, scales, block_ids, seqs: Seqs, block_size: int, softmax_scale=None,
                           out=None, lse=None, workspace=None):
    return _attn_fp8("decode", q, k, v, scales, block_ids, seqs, block_size, softmax_scale, out, lse, workspace)


# ---------------------------------------------------------------- dense baseline
def dense_attn_workspace_size(seqs: Seqs, num_q_heads: int, num_kv_heads: int, head_dim: int = 128) -> int:
    return int(lib().msa_dense_attn_workspace_size(seqs.ref(), num_q_heads, num_kv_heads, head_dim))


def dense_attn(q, k, v, seqs: Seqs, softmax_scale=None, out=None, lse=None, workspace=None):
    """Dense causal GQA attention (the baseline): (O bf16 [Tq, H_q, d], LSE fp32 [Tq, H_q])."""
    Tq, H_q, d_h = q.shape
    H_kv = k.shape[1]
    dev = seqs.device
    _need(q, "q", torch.bfloat16, (seqs.total_q_rows, H_q, d_h), dev)
    _need(k, "k", torch.bfloat16, (seqs.total_kv_rows, H_kv, d_h), dev)
    _need(v, "v", torch.bfloat16, (seqs.total_kv_rows, H_kv, d_h), dev)
    if out is None:
        out = torch.empty((Tq, H_q, d_h), dtype=torch.bfloat16, device=dev)
    if lse is None:
        lse = torch.empty((Tq, H_q), dtype=torch.float32, device=dev)
    _need(out, "o", torch.bfloat16, (Tq, H_q, d_h), dev)
    _need(lse, "lse", torch.float32, (Tq, H_q), dev)
    scale = 1.0 / math.sqrt(d_h) if softmax_scale is None else float(softmax_scale)
    nbytes = dense_attn_workspace_size(seqs, H_q, H_kv, d_h)
    ws = _workspace(nbytes, dev, workspace)
    st = lib().msa_dense_attn(_ptr(q), _ptr(k), _ptr(v), seqs.ref(), H_q, H_kv, d_h, scale, _ptr(out), _ptr(lse),
                              _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(), _stream())
    _check(st, "msa_dense_attn")
    return out, lse


# ---------------------------------------------------------------- kernel timing
# ---------------------------------------------------------------- training backward
def sparse_attn_backward_workspace_size(seqs: Seqs, num_q_heads, num_kv_heads, head_dim, block_size, topk) -> int:
    return int(lib().msa_sparse_attn_backward_workspace_size(seqs.ref(), num_q_heads, num_kv_heads, head_dim,
                                                              block_size, topk))


def sparse_attn_backward(q, k, v, o, lse, d_o, block_ids, seqs: Seqs, block_size: int, softmax_scale=None,
                         d_q=None, d_k=None, d_v=None, workspace=None):
    """dQ [Tq, H_q, d_h], dK and dV [Tkv, H_kv, d_h] (bf16) of the Main Branch for
    the upstream gradient d_o, given the forward's O and LSE."""
    Tq, H_q, d_h = q.shape
    H_kv = k.shape[1]
    topk = block_ids.shape[2]
    dev = seqs.device
    _need(q, "q", torch.bfloat16, (seqs.total_q_rows, H_q, d_h), dev)
    _need(k, "k", torch.bfloat16, (seqs.total_kv_rows, H_kv, d_h), dev)
    _need(v, "v", torch.bfloat16, (seqs.total_kv_rows, H_kv, d_h), dev)
    _need(o, "o", torch.bfloat16, (Tq, H_q, d_h), dev)
    _need(lse, "lse", torch.float32, (Tq, H_q), dev)
    _need(d_o, "d_o", torch.bfloat16, (Tq, H_q, d_h), dev)
    _need(block_ids, "block_ids", torch.int32, (Tq, H_kv, topk), dev)
    if d_q is None:
        d_q = torch.empty_like(q)
    if d_k is None:
        d_k = torch.empty_like(k)
    if d_v is None:
        d_v = torch.empty_like(v)
    _need(d_q, "d_q", torch.bfloat16, tuple(q.shape), dev)
    _need(d_k, "d_k", torch.bfloat16, tuple(k.shape), dev)
    _need(d_v, "d_v", torch.bfloat16, tuple(v.shape), dev)
    scale = 1.0 / math.sqrt(d_h) if softmax_scale is None else float(softmax_scale)
    L = lib()
    nbytes = int(L.msa_sparse_attn_backward_workspace_size(seqs.ref(), H_q, H_kv, d_h, block_size, topk))
    ws = _workspace(nbytes, dev, workspace)
    st = L.msa_sparse_attn_backward(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse), _ptr(d_o), _ptr(block_ids),
                                    seqs.ref(), H_q, H_kv, d_h, block_size, topk, scale, _ptr(d_q), _ptr(d_k),
                                    _ptr(d_v), _ptr(ws), 0 if ws is None else ws.numel() * ws.element_size(),
                                    _stream())
    _check(st, "msa_sparse_attn_backward")
    return d_q, d_k, d_v


def sparse_kl_backward_workspace_size(seqs: Seqs, num_q_heads, num_kv_heads, d_idx, head_dim, block_size,
                                      topk) -> int:
    return int(lib().msa_sparse_kl_backward_workspace_size(seqs.ref(), num_q_heads, num_kv_heads, d_idx, head_dim,
                                                            block_size, topk))


def sparse_kl_backward(index_q, index_k, q, k, lse, block_ids, seqs: Seqs, block_size: int, grad_scale: float = 1.0,
                       softmax_scale=None, with_kl: bool = True, d_index_q=None, d_index_k=None, kl=None,
                       workspace=None):
    """Sparse KL loss of the Index Branch: (d_index_q [Tq, H_kv, d_idx] bf16,
    d_index_k [Tkv, d_idx] bf16, kl [Tq, H_kv] fp32 or None); the gradients are
    grad_scale times those of sum(kl)."""
    Tq, H_kv, d_idx = index_q.shape
    H_q, d_h = q.shape[1], q.shape[2]
    topk = block_ids.shape[2]
    dev = seqs.device
    _need(index_q, "index_q", torch.bfloat16, (seqs.total_q_rows, H_kv, d_idx), dev)
    _need(index_k, "index_k", torch.bfloat16, (seqs.total_kv_rows, d_idx), dev)
    _need(q, "q", torch.bfloat16, (seqs.total_q_rows, H_q, d_h), dev)
    _need(k, "k", torch.bfloat16, (seqs.total_kv_rows, H_kv, d_h), dev)
    _need(lse, "lse", torch.float32, (Tq, H_q), dev)
    _need(block_ids, "block_ids", torch.int32, (Tq, H_kv, topk), dev)
    if d_index_q is None:
        d_index_q = torch.empty_like(index_q)
    if d_index_k is None:
        d_index_k = torch.empty_like(index_k)
    if with_kl and kl is None:
        kl = torch.empty((Tq, H_kv), dtype=torch.float32, device=dev)
    _need(d_index_q, "d_index_q", torch.bfloat16, tuple(index_q.shape), dev)
    _need(d_index_k, "d_index_k", torch.bfloat16, tuple(index_k.shape), dev)
    if kl is not None:
        _need(kl, "kl", torch.float32, (Tq, H_kv), dev)
    scale = 1.0 / math.sqrt(d_h) if softmax_scale is None else float(softmax_scale)
    L = lib()
    nbytes = int(L.msa_sparse_kl_backward_workspace_size(seqs.ref(), H_q, H_kv, d_idx, d_h, block_size, topk))
    ws = _workspace(nbytes, dev, workspace)
    st = L.msa_sparse_kl_backward(_ptr(index_q), _ptr(index_k), _ptr(q), _ptr(k), _ptr(lse), _ptr(block_ids),
                                  seqs.ref(), H_q, H_kv, d_idx, d_h, block_size, topk, scale, float(grad_scale),
                                  _ptr(d_index_q), _ptr(d_index_k), _ptr(kl), _ptr(ws),
                                  0 if ws is None else ws.numel() * ws.element_size(), _stream())
    _check(st, "msa_sparse_kl_backward")
    return d_index_q, d_index_k, kl


def profile_enable(on: bool = True) -> None:
    """Bracket every kernel of later calls with HIP events on its stream."""
    _check(lib().msa_profile_enable(1 if on else 0), "msa_profile_enable")


def profile_reset() -> None:
    _check(lib().msa_profile_reset(), "msa_profile_reset")


def profile_read() -> dict:
    """{kernel name: (launches, summed ms)} since the last reset (waits for the events)."""
    L = lib()
    out = {}
    i = 0
    while True:
        name = L.msa_profile_kernel_name(i)
        if name is None:
            break
        n = ctypes.c_int64(0)
        ms = ctypes.c_double(0.0)
        _check(L.msa_profile_read(name, ctypes.byref(n), ctypes.byref(ms)), "msa_profile_read")
        if n.value > 0:
            out[name.decode()] = (int(n.value), float(ms.value))
        i += 1
    return out

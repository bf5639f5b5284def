"""ctypes binding of ``libsparse_prefill.so``: one Python function per C entry point.

The functions take torch device tensors, check that each buffer has the
shape, dtype, device and contiguity the C ABI expects (the library itself
cannot see buffer sizes), and pass raw pointers plus the current HIP stream.
All arithmetic happens in the library's kernels; there is no fallback. If
the library is missing or cannot be loaded, every call raises.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsparse_prefill.so")

SP_DTYPE = {"f32": 0, "bf16": 1}
SP_AGG = {"max": 0, "sum": 1}
SP_OP = {"dense": 0, "oracle": 1, "indexer": 2, "topk": 3, "sparse": 4, "kl": 5,
         "project": 6, "indexer_topk": 7}
TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}
STATUS = {0: "SP_OK", -1: "SP_ERR_NULL", -2: "SP_ERR_SHAPE", -3: "SP_ERR_UNSUPPORTED",
          -4: "SP_ERR_WORKSPACE", -5: "SP_ERR_ALIGN", -6: "SP_ERR_NO_DEVICE",
          -7: "SP_ERR_ARCH", -8: "SP_ERR_HIP"}


class SpProblem(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "seq_len", "num_q_heads", "num_kv_heads", "head_dim", "index_dim", "topk", "block_q",
        "causal", "local_window", "agg", "relu", "dtype")] + [
        ("attn_scale", ctypes.c_float), ("index_scale", ctypes.c_float),
        ("head_axis", ctypes.c_int32), ("q_offset", ctypes.c_int32)]


@dataclasses.dataclass(frozen=True)
class Problem:
    """Python mirror of ``sp_problem`` (sizes as in the paper's Section 3)."""
    seq_len: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    index_dim: int = 0
    topk: int = 1
    block_q: int = 1
    causal: int = 1
    local_window: int = 0
    agg: str = "max"
    relu: bool = True
    dtype: str = "bf16"
    attn_scale: float = 0.0
    index_scale: float = 0.0
    head_axis: int = 0    # 1: one support per KV group (tables gain a leading Hkv axis)
    q_offset: int = 0     # chunked prefill: this call covers query positions q_offset..S-1

    @property
    def num_queries(self) -> int:
        return self.seq_len - self.q_offset

    @property
    def num_blocks(self) -> int:
        return (self.num_queries + self.block_q - 1) // self.block_q

    @property
    def table_rows(self) -> tuple:
        """Leading shape of mass/score and index tables."""
        R = self.num_blocks
        return (self.num_kv_heads, R) if self.head_axis else (R,)

    def to_c(self) -> SpProblem:
        return SpProblem(self.seq_len, self.num_q_heads, self.num_kv_heads, self.head_dim,
                         self.index_dim, self.topk, self.block_q, self.causal,
                         self.local_window, SP_AGG[self.agg], int(bool(self.relu)),
                         SP_DTYPE[self.dtype], self.attn_scale, self.index_scale,
                         int(self.head_axis), int(self.q_offset))


class SparsePrefillError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {STATUS.get(status, status)} ({status_string(status)})")


_lib = None


def lib_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Load the library (raises OSError/FileNotFoundError if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise FileNotFoundError(
                f"{_LIB_PATH} is missing: build it with `python -m paper_2606_07703_amd.build`")
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        PP = ctypes.POINTER(SpProblem)
        lib.sp_dense_attn.argtypes = [PP, P, P, P, P, P, P]
        lib.sp_oracle_support.argtypes = [PP, P, P, P, P, P]
        lib.sp_indexer_scores.argtypes = [PP, P, P, P, P]
        lib.sp_topk_select.argtypes = [PP, P, P, P, ctypes.c_size_t, P]
        lib.sp_sparse_gqa_attn.argtypes = [PP, P, P, P, P, P, P]
        lib.sp_kl_loss.argtypes = [PP, P, ctypes.c_int32, P, P, P, P, P, P]
        I32, F = ctypes.c_int32, ctypes.c_float
        lib.sp_indexer_project.argtypes = [PP, I32, I32, F, F, P, P, P, P, P, P, P, P]
        lib.sp_indexer_topk.argtypes = [PP, P, P, P, P, ctypes.c_size_t, P]
        lib.sp_indexer_topk_noalloc.argtypes = [PP, P, P, P, P]
        lib.sp_sparse_gqa_attn_paged.argtypes = [PP, P, P, P, P, I32, I32, P, P, P]
        lib.sp_workspace_bytes.argtypes = [PP, ctypes.c_int, ctypes.POINTER(ctypes.c_size_t)]
        lib.sp_status_string.argtypes = [ctypes.c_int]
        lib.sp_status_string.restype = ctypes.c_char_p
        lib.sp_version.argtypes = []
        for f in ("sp_dense_attn", "sp_oracle_support", "sp_indexer_scores", "sp_topk_select",
                  "sp_sparse_gqa_attn", "sp_kl_loss", "sp_indexer_project", "sp_indexer_topk",
                  "sp_indexer_topk_noalloc", "sp_sparse_gqa_attn_paged",
                  "sp_workspace_bytes", "sp_version"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def status_string(status: int) -> str:
    try:
        return load().sp_status_string(status).decode()
    except OSError:
        return STATUS.get(status, "unknown")


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return getattr(stream, "cuda_stream", stream)


def _ptr(t: Optional[torch.Tensor], name: str, shape, dtype) -> Optional[int]:
    if t is None:
        return None
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    return t.data_ptr()


def _call(fn: str, *args) -> None:
    rc = getattr(load(), fn)(*args)
    if rc != 0:
        raise SparsePrefillError(fn, rc)


def sp_dense_attn(p: Problem, q, k, v, o=None, lse=None, stream=None) -> None:
    S, Hq, Hkv, d = p.seq_len, p.num_q_heads, p.num_kv_heads, p.head_dim
    dt = TORCH_DTYPE[p.dtype]
    c = p.to_c()
    nq = p.num_queries
    _call("sp_dense_attn", ctypes.byref(c), _ptr(q, "q", (nq, Hq, d), dt),
          _ptr(k, "k", (S, Hkv, d), dt), _ptr(v, "v", (S, Hkv, d), dt),
          _ptr(o, "o", (nq, Hq, d), dt), _ptr(lse, "lse", (nq, Hq), torch.float32),
          _stream(stream))


def sp_oracle_support(p: Problem, q, k, lse, mass, stream=None) -> None:
    S, Hq, Hkv, d = p.seq_len, p.num_q_heads, p.num_kv_heads, p.head_dim
    dt = TORCH_DTYPE[p.dtype]
    c = p.to_c()
    _call("sp_oracle_support", ctypes.byref(c), _ptr(q, "q", (S, Hq, d), dt),
          _ptr(k, "k", (S, Hkv, d), dt), _ptr(lse, "lse", (S, Hq), torch.float32),
          _ptr(mass, "mass", p.table_rows + (S,), torch.float32), _stream(stream))


def sp_indexer_scores(p: Problem, q_idx, k_idx, scores, stream=None) -> None:
    S, di = p.seq_len, p.index_dim
    dt = TORCH_DTYPE[p.dtype]
    c = p.to_c()
    _call("sp_indexer_scores", ctypes.byref(c),
          _ptr(q_idx, "q_idx", (p.num_queries, di), dt),
          _ptr(k_idx, "k_idx", (S, di), dt),
          _ptr(scores, "scores", (p.num_blocks, S), torch.float32), _stream(stream))


def sp_topk_select(p: Problem, scores, idx, workspace=None, stream=None) -> None:
    c = p.to_c()
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    ws_ptr = None
    if workspace is not None:
        if workspace.device.type != "cuda" or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous device tensor")
        ws_ptr = workspace.data_ptr()
    _call("sp_topk_select", ctypes.byref(c),
          _ptr(scores, "scores", p.table_rows + (p.seq_len,), torch.float32),
          _ptr(idx, "idx", p.table_rows + (p.topk,), torch.int32), ws_ptr, ws_bytes,
          _stream(stream))


def sp_sparse_gqa_attn(p: Problem, q, k, v, idx, o, stream=None) -> None:
    S, Hq, Hkv, d = p.seq_len, p.num_q_heads, p.num_kv_heads, p.head_dim
    dt = TORCH_DTYPE[p.dtype]
    c = p.to_c()
    _call("sp_sparse_gqa_attn", ctypes.byref(c), _ptr(q, "q", (p.num_queries, Hq, d), dt),
          _ptr(k, "k", (S, Hkv, d), dt), _ptr(v, "v", (S, Hkv, d), dt),
          _ptr(idx, "idx", p.table_rows + (p.topk,), torch.int32),
          _ptr(o, "o", (p.num_queries, Hq, d), dt), _stream(stream))


def sp_indexer_topk(p: Problem, q_idx, k_idx, idx, workspace=None, stream=None) -> None:
    """Fused per-query indexer scores and top-k (no S x S score buffer).

    workspace: a device uint8 tensor of at least sp_workspace_bytes(p,
    "indexer_topk") bytes; when None one is taken from torch's allocator.
    """
    S, di = p.seq_len, p.index_dim
    need = sp_workspace_bytes(p, "indexer_topk")
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q_idx.device)
    nbytes = workspace.numel() * workspace.element_size()
    c = p.to_c()
    bf = torch.bfloat16
    _call("sp_indexer_topk", ctypes.byref(c), _ptr(q_idx, "q_idx", (S, di), bf),
          _ptr(k_idx, "k_idx", (S, di), bf), _ptr(idx, "idx", (S, p.topk), torch.int32),
          _ptr(workspace, "workspace", tuple(workspace.shape), workspace.dtype), nbytes,
          _stream(stream))


def sp_indexer_topk_noalloc(p: Problem, q_idx, k_idx, idx, stream=None) -> None:
    """sp_indexer_topk with its scratch in the library's static device array
    (no workspace; seq_len up to about 20480)."""
    S, di = p.seq_len, p.index_dim
    c = p.to_c()
    bf = torch.bfloat16
    _call("sp_indexer_topk_noalloc", ctypes.byref(c), _ptr(q_idx, "q_idx", (S, di), bf),
          _ptr(k_idx, "k_idx", (S, di), bf), _ptr(idx, "idx", (S, p.topk), torch.int32),
          _stream(stream))


def sp_indexer_project(p: Problem, x, w_q, w_k, gamma, beta, q_idx, k_idx, pos0: int = 0,
                       rope_theta: float = 10000.0, ln_eps: float = 1e-6, stream=None) -> None:
    """q_idx = RoPE(W_Q x), k_idx = RoPE(LN(W_K x)) at positions pos0 + t."""
    S, di = p.seq_len, p.index_dim
    dm = x.shape[1] if x is not None and x.dim() == 2 else 0
    c = p.to_c()
    bf = torch.bfloat16
    _call("sp_indexer_project", ctypes.byref(c), dm, pos0, rope_theta, ln_eps,
          _ptr(x, "x", (S, dm), bf), _ptr(w_q, "w_q", (di, dm), bf),
          _ptr(w_k, "w_k", (di, dm), bf), _ptr(gamma, "gamma", (di,), torch.float32),
          _ptr(beta, "beta", (di,), torch.float32), _ptr(q_idx, "q_idx", (S, di), bf),
          _ptr(k_idx, "k_idx", (S, di), bf), _stream(stream))


def sp_kl_loss(p: Problem, rows, P, z, kl=None, loss=None, grad_z=None, stream=None) -> None:
    """KL(P_i || softmax(z_i)) over s <= rows[i], the mean loss and its gradient."""
    S = p.seq_len
    n = rows.shape[0] if rows is not None else 0
    c = p.to_c()
    _call("sp_kl_loss", ctypes.byref(c), _ptr(rows, "rows", (n,), torch.int32), n,
          _ptr(P, "P", (n, S), torch.float32), _ptr(z, "z", (n, S), torch.float32),
          _ptr(kl, "kl", (n,), torch.float32), _ptr(loss, "loss", (1,), torch.float32),
          _ptr(grad_z, "grad_z", (n, S), torch.float32), _stream(stream))


def sp_sparse_gqa_attn_paged(p: Problem, q, k_pages, v_pages, page_table, idx, o,
                             stream=None) -> None:
    """Sparse GQA attention with K/V in a paged cache [num_pages, page_size, Hkv, d]."""
    S, Hq, Hkv, d = p.seq_len, p.num_q_heads, p.num_kv_heads, p.head_dim
    dt = TORCH_DTYPE[p.dtype]
    npg, ps = (k_pages.shape[0], k_pages.shape[1]) if k_pages is not None else (0, 0)
    c = p.to_c()
    _call("sp_sparse_gqa_attn_paged", ctypes.byref(c),
          _ptr(q, "q", (p.num_queries, Hq, d), dt),
          _ptr(k_pages, "k_pages", (npg, ps, Hkv, d), dt),
          _ptr(v_pages, "v_pages", (npg, ps, Hkv, d), dt),
          _ptr(page_table, "page_table", ((S + ps - 1) // max(ps, 1),), torch.int32), ps, npg,
          _ptr(idx, "idx", p.table_rows + (p.topk,), torch.int32),
          _ptr(o, "o", (p.num_queries, Hq, d), dt), _stream(stream))


def sp_workspace_bytes(p: Problem, op: str) -> int:
    c = p.to_c()
    n = ctypes.c_size_t(0)
    _call("sp_workspace_bytes", ctypes.byref(c), SP_OP[op], ctypes.byref(n))
    return n.value


def sp_version() -> int:
    return load().sp_version()

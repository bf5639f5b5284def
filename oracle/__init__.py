"""fp64 CPU oracle for causal top-k sparse GQA prefill (test infrastructure).

Only the tests, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package. It shares no code with the GPU library and never
takes an input produced by it.

The C library (``sp_oracle.c``) holds the paper's definitions, written plainly
in double precision; this module marshals numpy arrays and composes the steps
in the paper's order:

* oracle mode (Algorithm 1): dense normalisers -> head-averaged mass P ->
  block aggregation -> top-k -> restricted attention;
* indexer mode (Algorithm 2, scoring, selection and sparse prefill): indexer scores -> block aggregation
  -> top-k -> restricted attention;
* dense attention (Section 3);
* the KL distillation objective and its gradient (Section 6.2);
* the head-collapsed indexer front end: projection, key LayerNorm, RoPE
  (Section 6.3, Algorithm 2, indexer projection and its key normalisation, RoPE and query scale).

Parity pins for every function live in ``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "sp_oracle.c")
_LIB = os.path.join(_HERE, "libsp_oracle.so")
# A prebuilt copy of the same source to load instead (the sanitizer test
# builds one with AddressSanitizer and UBSan); it is used as it is.
_LIB_OVERRIDE = os.environ.get("SP_ORACLE_LIB")
_lib = None

AGG = {"max": 0, "sum": 1}


def build(force: bool = True) -> str:
    """Compile the oracle's C source with gcc (OpenMP, portable -O2)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            lib = ctypes.CDLL(_LIB_OVERRIDE)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        D = ctypes.c_double
        lib.orc_dense.argtypes = [I, I, I, I, D, P, P, P, I, P, P, P]
        lib.orc_mass.argtypes = [I, I, I, I, D, P, P, I, P, P]
        lib.orc_index_scores.argtypes = [I, I, D, I, P, P, I, P, P]
        lib.orc_block_aggregate.argtypes = [I, I, I, P, P, P]
        lib.orc_topk.argtypes = [I, P, P, ctypes.c_int64, I, I, P]
        lib.orc_sparse.argtypes = [I, I, I, I, D, P, P, P, I, I, P, ctypes.c_int64, I, P, P]
        lib.orc_mass_heads.argtypes = [I, I, I, I, D, P, P, I, I, I, P, P]
        lib.orc_kl.argtypes = [I, I, P, P, P, P, P]
        lib.orc_project.argtypes = [I, I, I, P, P, P, P, P, D, D, I, I, P, P, P]
        lib.orc_num_threads.argtypes = []
        lib.orc_num_threads.restype = ctypes.c_int
        for f in ("orc_dense", "orc_mass", "orc_index_scores", "orc_block_aggregate",
                  "orc_topk", "orc_sparse", "orc_kl", "orc_project", "orc_mass_heads"):
            getattr(lib, f).restype = None
        _lib = lib
    return _lib


def num_threads() -> int:
    """Threads the oracle's OpenMP loops use on this host."""
    return int(_load().orc_num_threads())


def _f64(a) -> np.ndarray:
    """Widen (exactly) to a contiguous float64 numpy array. Accepts torch CPU tensors."""
    if hasattr(a, "detach"):
        a = a.detach().to("cpu")
        import torch
        a = a.to(torch.float64).numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _i32(a) -> np.ndarray:
    if hasattr(a, "detach"):
        a = a.detach().to("cpu").numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _rows(S: int, rows) -> np.ndarray:
    return _i32(np.arange(S) if rows is None else rows)


def block_rows(S: int, b: int, r: int) -> np.ndarray:
    """Query positions of selection block r: [r*b, min(r*b+b, S))."""
    return np.arange(r * b, min(r * b + b, S), dtype=np.int32)


def num_blocks(S: int, b: int) -> int:
    return (S + b - 1) // b


# ---------------------------------------------------------------- primitives
def dense(q, k, v, rows=None, scale: Optional[float] = None, want_o: bool = True):
    """Dense causal GQA attention rows (Section 3). Returns (o [n,Hq,d], lse [n,Hq])."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    S, Hq, d = q.shape
    Hkv = k.shape[1]
    rows = _rows(S, rows)
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    o = np.zeros((len(rows), Hq, d)) if want_o else None
    lse = np.zeros((len(rows), Hq))
    _load().orc_dense(S, Hq, Hkv, d, scale, _ptr(q), _ptr(k), _ptr(v), len(rows),
                      _ptr(rows), _ptr(o), _ptr(lse))
    return o, lse


def mass(q, k, rows=None, scale: Optional[float] = None, group: Optional[int] = None) -> np.ndarray:
    """Head-averaged attention mass rows P_t(s) (Section 4.1). Returns [n,S].

    group=None averages over every query head (the token support S_t);
    group=j over the G heads of KV group j (the per-group support S_{t,j}).
    """
    q, k = _f64(q), _f64(k)
    S, Hq, d = q.shape
    Hkv = k.shape[1]
    rows = _rows(S, rows)
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    P = np.zeros((len(rows), S))
    if group is None:
        _load().orc_mass(S, Hq, Hkv, d, scale, _ptr(q), _ptr(k), len(rows), _ptr(rows), _ptr(P))
    else:
        G = Hq // Hkv
        _load().orc_mass_heads(S, Hq, Hkv, d, scale, _ptr(q), _ptr(k), group * G, G, len(rows),
                               _ptr(rows), _ptr(P))
    return P


def index_scores(q_idx, k_idx, rows=None, scale: Optional[float] = None,
                 relu: bool = True) -> np.ndarray:
    """Indexer scores z[t,s] (Section 6.3). Returns [n,S]."""
    qi, ki = _f64(q_idx), _f64(k_idx)
    S, di = qi.shape
    rows = _rows(S, rows)
    scale = 1.0 / np.sqrt(di) if scale is None else scale
    Z = np.zeros((len(rows), S))
    _load().orc_index_scores(S, di, scale, int(relu), _ptr(qi), _ptr(ki), len(rows),
                             _ptr(rows), _ptr(Z))
    return Z


def aggregate(X: np.ndarray, trows, agg: str = "max") -> np.ndarray:
    """Block aggregate of per-query rows X [nt,S] (Section 4.2). Returns [S]."""
    X = _f64(X)
    trows = _i32(trows)
    S = X.shape[1]
    Y = np.zeros(S)
    _load().orc_block_aggregate(S, AGG[agg], len(trows), _ptr(trows), _ptr(X), _ptr(Y))
    return Y


def topk(Y: np.ndarray, lens, k: int, window: int = 0) -> np.ndarray:
    """Top-k supports of score rows Y [n,>=max(lens)] (Section 4.1, Algorithm 1, selection and restricted recomputation)."""
    Y = _f64(np.atleast_2d(Y))
    lens = _i32(np.atleast_1d(lens))
    out = np.full((len(lens), k), -1, dtype=np.int32)
    _load().orc_topk(len(lens), _ptr(lens), _ptr(Y), Y.shape[1], k, window, _ptr(out))
    return out


def sparse(q, k, v, idx, block_q: int, rows=None, scale: Optional[float] = None) -> np.ndarray:
    """Restricted attention over supports (Section 3, 4.2). Returns [n,Hq,d].

    idx [R,kk]: one support per selection block shared by every head;
    idx [Hkv,R,kk]: one support per KV group, used by that group's heads.
    """
    q, k, v = _f64(q), _f64(k), _f64(v)
    idx = _i32(idx)
    S, Hq, d = q.shape
    Hkv = k.shape[1]
    rows = _rows(S, rows)
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    o = np.zeros((len(rows), Hq, d))
    stride = idx.shape[1] * idx.shape[2] if idx.ndim == 3 else 0
    if idx.ndim == 3:
        assert idx.shape[0] == Hkv
    _load().orc_sparse(S, Hq, Hkv, d, scale, _ptr(q), _ptr(k), _ptr(v), block_q,
                       idx.shape[-1], _ptr(idx), stride, len(rows), _ptr(rows), _ptr(o))
    return o


def sparse_paged(q, k_pages, v_pages, page_table, idx, block_q: int, rows=None,
                 scale: Optional[float] = None) -> np.ndarray:
    """Restricted attention with K/V in a paged cache (Section 6.4).

    Token s is row s % page_size of page page_table[s // page_size]; a
    selected position whose page entry lies outside the cache contributes
    nothing (it becomes a sentinel). The attention itself is ``sparse``.
    """
    kp, vp = _f64(k_pages), _f64(v_pages)
    table = _i32(page_table)
    idx = _i32(idx).copy()
    npg, ps = kp.shape[0], kp.shape[1]
    S = _f64(q).shape[0]
    k = np.zeros((S,) + kp.shape[2:])
    v = np.zeros((S,) + vp.shape[2:])
    ok = np.zeros(S, dtype=bool)
    for s in range(S):
        pg = table[s // ps]
        if 0 <= pg < npg:
            k[s], v[s], ok[s] = kp[pg, s % ps], vp[pg, s % ps], True
    valid = (idx >= 0) & (idx < S)
    bad = valid & ~ok[np.clip(idx, 0, S - 1)]
    idx[bad] = -1
    return sparse(q, k, v, idx, block_q, rows=rows, scale=scale)


def kl(P, z, rows):
    """KL(P_i || softmax(z_i)) over s <= rows[i] (Section 6.2).

    P, z are [n,S]. Returns (kl [n], grad [n,S]) where grad is the gradient of
    the mean over rows, L = (1/n) sum_i kl[i], with respect to z.
    """
    P, z = _f64(P), _f64(z)
    rows = _i32(rows)
    n, S = P.shape
    out = np.zeros(n)
    grad = np.zeros((n, S))
    _load().orc_kl(S, n, _ptr(rows), _ptr(P), _ptr(z), _ptr(out), _ptr(grad))
    return out, grad


def project(x, wq, wk, gamma, beta, rows=None, pos0: int = 0, theta: float = 10000.0,
            eps: float = 1e-6):
    """Indexer front end (Section 6.3; Algorithm 2, indexer projection and its key normalisation, RoPE and query scale).

    x [S,dm], wq/wk [d_idx,dm], gamma/beta [d_idx]. Returns (q_idx, k_idx),
    each [n,d_idx]: RoPE(W_Q x_t) and RoPE(LN(W_K x_t)) at positions pos0 + t.
    """
    x, wq, wk = _f64(x), _f64(wq), _f64(wk)
    gamma, beta = _f64(gamma), _f64(beta)
    S, dm = x.shape
    di = wq.shape[0]
    rows = _rows(S, rows)
    qo = np.zeros((len(rows), di))
    ko = np.zeros((len(rows), di))
    _load().orc_project(S, dm, di, _ptr(x), _ptr(wq), _ptr(wk), _ptr(gamma), _ptr(beta),
                        eps, theta, pos0, len(rows), _ptr(rows), _ptr(qo), _ptr(ko))
    return qo, ko


# ----------------------------------------------------------------- pipelines
def support_scores(mode: str, units: Sequence[int], block_q: int, *, q=None, k=None,
                   q_idx=None, k_idx=None, agg: str = "max", attn_scale=None,
                   index_scale=None, relu: bool = True, group: Optional[int] = None) -> np.ndarray:
    """Aggregated score rows Y [len(units), S] for selection blocks ``units``.

    mode "oracle": X = head-averaged mass P (Algorithm 1, normalisers and head-averaged probabilities), over the
    heads of KV group ``group`` when given (per-group support);
    mode "indexer": X = indexer scores z (Algorithm 2, candidate scoring).
    Then Y = block aggregate of X (identity when block_q == 1).
    """
    S = (q if mode == "oracle" else q_idx).shape[0]
    out = np.zeros((len(units), S))
    for n, r in enumerate(units):
        trows = block_rows(S, block_q, r)
        if mode == "oracle":
            X = mass(q, k, trows, attn_scale, group=group)
        elif mode == "indexer":
            X = index_scores(q_idx, k_idx, trows, index_scale, relu)
        else:
            raise ValueError(mode)
        out[n] = X[0] if len(trows) == 1 else aggregate(X, trows, agg)
    return out


def select(Y: np.ndarray, units: Sequence[int], block_q: int, S: int, k: int,
           window: int = 0) -> np.ndarray:
    """Top-k of aggregated rows; row of unit r has t1_r+1 valid positions."""
    lens = np.array([min(r * block_q + block_q, S) for r in units], dtype=np.int32)
    return topk(Y, lens, k, window)


def topk_gap(Y: np.ndarray, L: int, k: int, window: int = 0):
    """(v_k, v_{k+1}, relative gap) among the non-forced candidates of one row.

    Used by the parity rule for selected sets: sets must agree exactly where
    the gap between the k'-th and (k'+1)-th candidate values exceeds 1e-4
    relative. Returns None when the row has at most k valid positions.
    """
    if L <= k:
        return None
    Wf = min(window, k)
    kp = k - Wf
    c = np.sort(np.asarray(Y[: L - Wf], dtype=np.float64))[::-1]
    if kp == 0:
        return None
    vk, vk1 = c[kp - 1], c[kp]
    return vk, vk1, (vk - vk1) / max(abs(vk), 1e-30)

"""The C ABI on the host: loading, exported symbols, argument validation.

Validation runs before any HIP call, so every status here is reachable
without a GPU. No compute entry point is launched on a device.
"""
import ctypes
import os
import re

import pytest
import torch

from paper_2606_07703_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparse_prefill.h")
NO_DEVICE = torch.cuda.device_count() == 0

OK, NULL, SHAPE, UNSUP, WS, ALIGN, NODEV, ARCH, HIP = 0, -1, -2, -3, -4, -5, -6, -7, -8
A, A2, A3, A4, A5, A6 = 0x10000, 0x20000, 0x30000, 0x40000, 0x50000, 0x60000  # never dereferenced


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sp_[a-z_]+)\s*\(", text)))


def lib():
    return B.load()


def prob(**kw):
    base = dict(seq_len=128, num_q_heads=8, num_kv_heads=2, head_dim=128, index_dim=64,
                topk=16, block_q=4, dtype="bf16")
    base.update(kw)
    return B.Problem(**base).to_c()


def test_library_exports_every_declared_symbol():
    names = declared_symbols()
    assert set(names) >= {"sp_dense_attn", "sp_oracle_support", "sp_indexer_scores",
                          "sp_topk_select", "sp_sparse_gqa_attn", "sp_workspace_bytes",
                          "sp_status_string", "sp_version"}
    L = lib()
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_strings():
    assert B.sp_version() == 10000
    for s in (OK, NULL, SHAPE, UNSUP, WS, ALIGN, NODEV, ARCH, HIP):
        assert B.status_string(s) not in ("", "unknown status")
    assert B.status_string(123) == "unknown status"


def rc(fn, p, *args):
    return getattr(lib(), fn)(ctypes.byref(p) if p is not None else None, *args)


def dense(p, q=A, k=A2, v=A3, o=A4, lse=A5):
    return rc("sp_dense_attn", p, q, k, v, o, lse, None)


def sparse(p, q=A, k=A2, v=A3, idx=A4, o=A5):
    return rc("sp_sparse_gqa_attn", p, q, k, v, idx, o, None)


def indexer(p, qi=A, ki=A2, sc=A3):
    return rc("sp_indexer_scores", p, qi, ki, sc, None)


def topk(p, sc=A, idx=A2, ws=None, nbytes=0):
    return rc("sp_topk_select", p, sc, idx, ws, nbytes, None)


def oracle_support(p, q=A, k=A2, lse=A3, mass=A4):
    return rc("sp_oracle_support", p, q, k, lse, mass, None)


def test_null_pointers():
    assert dense(None) == NULL
    assert dense(prob(), q=None) == NULL
    assert dense(prob(), o=None, lse=None) == NULL
    assert sparse(prob(), idx=None) == NULL
    assert indexer(prob(), sc=None) == NULL
    assert topk(prob(), idx=None) == NULL
    assert oracle_support(prob(), lse=None) == NULL
    n = ctypes.c_size_t()
    assert lib().sp_workspace_bytes(None, 0, ctypes.byref(n)) == NULL


@pytest.mark.parametrize("kw,expect", [
    (dict(seq_len=0), SHAPE),
    (dict(num_q_heads=6, num_kv_heads=4), SHAPE),
    (dict(num_kv_heads=0), SHAPE),
    (dict(head_dim=96), UNSUP),
    (dict(causal=0), UNSUP),
    (dict(num_q_heads=512, num_kv_heads=2), UNSUP),
    # k and v of 4 GiB each (rows are addressed with 32-bit byte offsets)
    (dict(seq_len=1 << 21, num_q_heads=8, num_kv_heads=8, head_dim=128, dtype="bf16"), UNSUP),
])
def test_shape_errors_attention(kw, expect):
    assert dense(prob(**kw)) == expect
    assert sparse(prob(**kw)) == expect


@pytest.mark.parametrize("kw,expect", [
    (dict(topk=0), SHAPE),
    (dict(block_q=0), SHAPE),
    (dict(local_window=-1), SHAPE),
    (dict(local_window=17), SHAPE),
])
def test_selection_errors(kw, expect):
    assert sparse(prob(**kw)) == expect
    assert topk(prob(**kw)) == expect
    assert indexer(prob(**kw)) == expect
    assert oracle_support(prob(**kw)) == expect


@pytest.mark.parametrize("scale", [-0.088, -1e-30, float("nan"), float("inf")])
def test_attention_scale_must_be_positive_and_finite(scale):
    # the MFMA attention kernels take row maxima of raw scores and scale them
    # afterwards, which only commutes with the max for a positive scale
    p = prob(attn_scale=scale)
    assert dense(p) == SHAPE and sparse(p) == SHAPE and oracle_support(p) == SHAPE
    assert rc("sp_sparse_gqa_attn_paged", p, A, A2, A3, A4, 64, 4, A5, A6, None) == SHAPE


def test_indexer_specific_errors():
    assert indexer(prob(index_dim=96)) == UNSUP
    assert indexer(prob(index_dim=0)) == UNSUP
    p = prob()
    p.agg = 7
    assert indexer(p) == SHAPE and oracle_support(p) == SHAPE
    p = prob()
    p.relu = 2
    assert indexer(p) == SHAPE
    p = prob()
    p.dtype = 9
    assert indexer(p) == UNSUP and dense(p) == UNSUP


def test_alignment():
    assert dense(prob(), q=A + 8) == ALIGN
    assert sparse(prob(), idx=A4 + 4) == ALIGN
    assert topk(prob(), sc=A + 2) == ALIGN
    assert indexer(prob(), ki=A2 + 6) == ALIGN


def test_workspace_query():
    for op in range(5):
        assert B.sp_workspace_bytes(B.Problem(128, 8, 2, 128, 64, 16, 4), list(B.SP_OP)[op]) == 0
    n = ctypes.c_size_t()
    assert lib().sp_workspace_bytes(ctypes.byref(prob()), 9, ctypes.byref(n)) == SHAPE


@pytest.mark.skipif(not NO_DEVICE, reason="checks the no-device path")
def test_valid_arguments_report_no_device():
    assert dense(prob()) == NODEV
    assert dense(prob(), o=None) == NODEV      # normaliser-only form is valid
    assert sparse(prob()) == NODEV
    assert indexer(prob()) == NODEV
    assert topk(prob()) == NODEV
    assert oracle_support(prob()) == NODEV
    with pytest.raises(B.SparsePrefillError):
        B._call("sp_topk_select", ctypes.byref(prob()), A, A2, None, 0, None)


def test_binding_rejects_bad_tensors():
    p = B.Problem(16, 4, 2, 64, dtype="f32", topk=4)
    cpu = torch.zeros(16, 4, 64)
    with pytest.raises(ValueError):
        B.sp_dense_attn(p, cpu, cpu, cpu, cpu)


def _project_args(**kw):
    a = dict(d_model=128, pos0=0, theta=10000.0, eps=1e-6)
    a.update(kw)
    pc = prob(index_dim=a.pop("index_dim", 64), dtype=a.pop("dtype", "bf16"))
    P = ctypes.c_void_p
    buf = [P(16)] * 7
    nulls = a.pop("nulls", ())
    for i in nulls:
        buf[i] = None
    return (ctypes.byref(pc), a["d_model"], a["pos0"], ctypes.c_float(a["theta"]),
            ctypes.c_float(a["eps"]), *buf, None)


@pytest.mark.parametrize("kw,expect", [
    (dict(d_model=96), UNSUP),
    (dict(index_dim=96), UNSUP),
    (dict(dtype="f32"), UNSUP),
    (dict(pos0=-1), SHAPE),
    (dict(theta=0.0), SHAPE),
    (dict(eps=-1.0), SHAPE),
    (dict(d_model=0), SHAPE),
    (dict(nulls=(3,)), NULL),
])
def test_project_errors(kw, expect):
    assert lib().sp_indexer_project(*_project_args(**kw)) == expect


def test_project_valid_arguments_report_no_device():
    if not NO_DEVICE:
        pytest.skip("a device is present")
    assert lib().sp_indexer_project(*_project_args()) == NODEV


def test_kl_errors():
    P = ctypes.c_void_p
    pc = prob()
    f = lib().sp_kl_loss
    assert f(None, P(16), 1, P(16), P(16), None, None, None, None) == NULL
    assert f(ctypes.byref(pc), P(16), -1, P(16), P(16), None, None, None, None) == SHAPE
    assert f(ctypes.byref(pc), P(16), 0, None, None, None, None, None, None) == 0   # no rows
    assert f(ctypes.byref(pc), P(16), 2, None, P(16), None, None, None, None) == NULL
    # the mean needs the per-row values
    assert f(ctypes.byref(pc), P(16), 2, P(16), P(16), None, P(16), None, None) == NULL
    assert f(ctypes.byref(pc), P(16), 2, P(16), P(18), None, None, None, None) == ALIGN
    if NO_DEVICE:
        assert f(ctypes.byref(pc), P(16), 2, P(16), P(16), P(16), P(16), P(16), None) == NODEV


@pytest.mark.parametrize("kw,expect", [
    (dict(q_offset=-1), SHAPE),
    (dict(q_offset=128), SHAPE),           # no query rows left (S = 128)
    (dict(q_offset=6, block_q=4), SHAPE),  # a chunk starts on a selection-block boundary
    (dict(head_axis=2), SHAPE),
])
def test_chunk_and_head_axis_errors(kw, expect):
    assert sparse(prob(**kw)) == expect
    assert topk(prob(**kw)) == expect


def test_oracle_support_and_fused_reject_chunks():
    assert oracle_support(prob(q_offset=8)) == UNSUP
    p = prob(q_offset=8, block_q=1)
    n = ctypes.c_size_t()
    assert lib().sp_indexer_topk(ctypes.byref(p), A, A2, A3, A4, 1 << 30, None) == UNSUP


def test_noalloc_refuses_problems_beyond_its_static_scratch():
    # about 20480 tokens fit the 64 MiB array; refused before any device call
    p = prob(seq_len=30000, block_q=1, index_dim=128, topk=64)
    assert rc("sp_indexer_topk_noalloc", p, A, A2, A3, None) == WS
    p = prob(seq_len=30000, block_q=4, index_dim=128, topk=64)
    assert rc("sp_indexer_topk_noalloc", p, A, A2, A3, None) == UNSUP
    assert rc("sp_indexer_topk_noalloc", prob(block_q=1), None, A2, A3, None) == NULL
    if NO_DEVICE:
        assert rc("sp_indexer_topk_noalloc", prob(block_q=1), A, A2, A3, None) == NODEV

"""GPU parity of the NEXT-row entry points against the fp64 oracle.

KL distillation loss (sp_kl_loss), the indexer front end
(sp_indexer_project) and the fused per-query indexer top-k (sp_indexer_topk). Inputs come from the seeded generators only; full-size
runs are checked on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_07703_amd import binding as B
from synth import make_index_vectors, make_inputs, make_kl_rows, make_projection_inputs

from helpers import check_rows_ascending, compare_support, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()


# The kernel sums P (log P - z) and P in fp64 and the exp-sum in fp32 with a
# running max; log and exp are fp32 (relative error a few 1e-7, growing with
# |z - LSE| through the argument rounding). Bounds below leave a 10x margin.
def _check_kl(kl, grad, loss, ref_kl, ref_grad, ref_loss=None):
    ekl = np.abs(kl - ref_kl) - (1e-4 + 1e-5 * np.abs(ref_kl))
    assert np.all(ekl <= 0), f"kl err {np.max(np.abs(kl - ref_kl)):.3e}"
    scale = np.maximum(np.max(np.abs(ref_grad), axis=1, keepdims=True), 1e-30)
    assert np.all(np.abs(grad - ref_grad) <= 1e-5 * scale), \
        f"grad err {np.max(np.abs(grad - ref_grad) / scale):.3e} of row max"
    if ref_loss is not None:
        assert abs(loss - ref_loss) <= 1e-4 + 1e-5 * abs(ref_loss)


@pytest.mark.parametrize("n,S,zero_frac", [(1, 1, 0.0), (50, 300, 0.0), (64, 1000, 0.4),
                                           (7, 33, 0.9)])
def test_kl_loss(n, S, zero_frac):
    say(f"kl n={n} S={S} zero_frac={zero_frac}")
    t = np.random.default_rng(n + S).integers(0, S, size=n)
    t[0] = S - 1
    rows, P, z = make_kl_rows(n, S, seed=n + S, rows=t, zero_frac=zero_frac)
    p = B.Problem(S, 1, 1, 64)
    kl = torch.empty(n, device="cuda")
    loss = torch.empty(1, device="cuda")
    grad = torch.full((n, S), 7.0, device="cuda")
    B.sp_kl_loss(p, rows.cuda(), P.cuda(), z.cuda(), kl, loss, grad)
    torch.cuda.synchronize()
    ref_kl, ref_grad = oracle.kl(P.numpy(), z.numpy(), rows.numpy())
    _check_kl(kl.cpu().double().numpy(), grad.cpu().double().numpy(), loss.item(),
              ref_kl, ref_grad, ref_kl.mean())


def test_kl_loss_long_rows_and_invalid_rows():
    S = 40000   # rows longer than the register-resident limit stream twice
    rows = torch.tensor([S - 1, 32767, 32768, 5, -1, S], dtype=torch.int32)
    _, P, z = make_kl_rows(6, S, seed=3, rows=rows.clamp(0, S - 1), zero_frac=0.1)
    p = B.Problem(S, 1, 1, 64)
    kl = torch.empty(6, device="cuda")
    grad = torch.full((6, S), 7.0, device="cuda")
    B.sp_kl_loss(p, rows.cuda(), P.cuda(), z.cuda(), kl, None, grad)
    torch.cuda.synchronize()
    ref_kl, ref_grad = oracle.kl(P.numpy(), z.numpy(), rows.numpy())
    assert ref_kl[4] == 0.0 and ref_kl[5] == 0.0
    _check_kl(kl.cpu().double().numpy(), grad.cpu().double().numpy(), None, ref_kl, ref_grad)


def test_kl_loss_optional_outputs():
    S, n = 200, 9
    rows, P, z = make_kl_rows(n, S, seed=9)
    p = B.Problem(S, 1, 1, 64)
    rc, Pc, zc = rows.cuda(), P.cuda(), z.cuda()
    grad = torch.empty(n, S, device="cuda")
    B.sp_kl_loss(p, rc, Pc, zc, None, None, grad)          # gradient only
    kl = torch.empty(n, device="cuda")
    B.sp_kl_loss(p, rc, Pc, zc, kl, None, None)            # values only
    torch.cuda.synchronize()
    ref_kl, ref_grad = oracle.kl(P.numpy(), z.numpy(), rows.numpy())
    _check_kl(kl.cpu().double().numpy(), grad.cpu().double().numpy(), None, ref_kl, ref_grad)
    with pytest.raises(B.SparsePrefillError):
        B.sp_kl_loss(p, rc, Pc, zc, None, torch.empty(1, device="cuda"), None)
    B.sp_kl_loss(p, rc[:0], Pc[:0], zc[:0])                 # no rows: a no-op


def test_kl_loss_full_size_sampled():
    S = 32768
    say(f"kl full size S={S}, every query row")
    rows, P, z = make_kl_rows(S, S, seed=4, rows=torch.arange(S), zero_frac=0.2,
                              device="cuda")
    p = B.Problem(S, 1, 1, 64)
    kl = torch.empty(S, device="cuda")
    loss = torch.empty(1, device="cuda")
    grad = torch.empty(S, S, device="cuda")
    B.sp_kl_loss(p, rows, P, z, kl, loss, grad)
    torch.cuda.synchronize()
    sample = np.array([0, 1, 2047, 4096, 16383, 30000, 32766, 32767])
    Ps, zs = P[sample].cpu().numpy(), z[sample].cpu().numpy()
    ref_kl, ref_grad = oracle.kl(Ps, zs, sample)
    # the oracle's gradient is of the mean over its own rows; rescale to S rows
    ref_grad *= len(sample) / S
    _check_kl(kl[sample].cpu().double().numpy(), grad[sample].cpu().double().numpy(), None,
              ref_kl, ref_grad)
    # the mean: fp64 sum of the kernel's own per-row values
    assert loss.item() == pytest.approx(kl.double().mean().item(), rel=1e-6)


# ---------------------------------------------------------------- front end
# Outputs are bf16 (round-to-nearest-even: relative error <= 2^-9) of values the
# kernel forms in fp32 from the same bf16 inputs the oracle reads exactly; the
# fp32 GEMM, LayerNorm and rotation add errors near 1e-6. Bound: 2^-8 relative
# plus 1e-4 absolute.
def _check_proj(got, ref):
    got = got.float().cpu().double().numpy()
    err = np.abs(got - ref) - (2.0 ** -8 * np.abs(ref) + 1e-4)
    assert np.all(err <= 0), f"max excess {err.max():.3e}, max abs err {np.abs(got - ref).max():.3e}"


def _project(S, dm, di, pos0, seed, theta=10000.0, eps=1e-6):
    x, wq, wk, gamma, beta = make_projection_inputs(S, dm, di, seed=seed)
    p = B.Problem(S, 1, 1, 64, index_dim=di)
    qo = torch.empty(S, di, dtype=torch.bfloat16, device="cuda")
    ko = torch.empty(S, di, dtype=torch.bfloat16, device="cuda")
    B.sp_indexer_project(p, x.cuda(), wq.cuda(), wk.cuda(), gamma.cuda(), beta.cuda(), qo, ko,
                         pos0=pos0, rope_theta=theta, ln_eps=eps)
    torch.cuda.synchronize()
    return (x, wq, wk, gamma, beta), qo, ko


@pytest.mark.parametrize("S,dm,di,pos0", [(1, 64, 64, 0), (130, 128, 64, 0),
                                          (130, 192, 128, 1000), (65, 256, 256, 7),
                                          (200, 512, 128, 100000), (300, 1024, 64, 5),
                                          (385, 4096, 128, 0), (129, 64, 128, 0),
                                          (257, 128, 128, 9)])
def test_indexer_project(S, dm, di, pos0):
    say(f"project S={S} d_model={dm} d_idx={di} pos0={pos0}")
    (x, wq, wk, gamma, beta), qo, ko = _project(S, dm, di, pos0, seed=S + di)
    rq, rk = oracle.project(x, wq, wk, gamma, beta, pos0=pos0)
    _check_proj(qo, rq)
    _check_proj(ko, rk)


def test_indexer_project_theta_and_eps():
    S, dm, di = 70, 128, 128
    (x, wq, wk, gamma, beta), qo, ko = _project(S, dm, di, 3, seed=1, theta=500000.0, eps=1e-3)
    rq, rk = oracle.project(x, wq, wk, gamma, beta, pos0=3, theta=500000.0, eps=1e-3)
    _check_proj(qo, rq)
    _check_proj(ko, rk)


def test_indexer_project_full_size_sampled():
    S, dm, di = 32768, 4096, 128
    say(f"project full size S={S} d_model={dm} d_idx={di}")
    (x, wq, wk, gamma, beta), qo, ko = _project(S, dm, di, 0, seed=4)
    sample = np.array([0, 1, 63, 64, 127, 128, 255, 4095, 20000, 32640, 32704, 32767])
    rq, rk = oracle.project(x, wq, wk, gamma, beta, rows=sample)
    _check_proj(qo[sample], rq)
    _check_proj(ko[sample], rk)


# ------------------------------------------------------- fused indexer top-k
def _fused_and_unfused(S, di, k, W, relu, qi, ki):
    p = B.Problem(S, 1, 1, 64, index_dim=di, topk=k, block_q=1, local_window=W, relu=relu)
    q, kk = qi.cuda(), ki.cuda()
    fused = torch.full((S, k), -7, dtype=torch.int32, device="cuda")
    B.sp_indexer_topk(p, q, kk, fused)
    sc = torch.empty(S, S, device="cuda")
    B.sp_indexer_scores(p, q, kk, sc)
    unfused = torch.empty(S, k, dtype=torch.int32, device="cuda")
    B.sp_topk_select(p, sc, unfused)
    torch.cuda.synchronize()
    return fused.cpu().numpy(), unfused.cpu().numpy()


FUSED_CASES = [
    # S, d_idx, k, W, relu, kind
    (1, 64, 4, 0, 1, "gauss"),
    (50, 128, 64, 0, 1, "gauss"),        # every row has L <= k
    (300, 64, 37, 0, 1, "gauss"),
    (300, 128, 37, 5, 0, "gauss"),
    (1000, 256, 100, 0, 1, "ternary"),   # integer scores: exact ties everywhere
    (5000, 128, 512, 0, 1, "gauss"),     # two key chunks
    (9000, 64, 256, 16, 1, "ternary"),   # three chunks, forced window, ties
    (700, 128, 700, 3, 1, "gauss"),      # k above every row length but the last
    (400, 128, 9, 9, 1, "gauss"),        # window takes the whole budget
]


@pytest.mark.parametrize("case", FUSED_CASES, ids=lambda c: "-".join(map(str, c)))
def test_indexer_topk_fused(case):
    S, di, k, W, relu, kind = case
    say(f"fused indexer top-k {case}")
    qi, ki = make_index_vectors(S, di, seed=S + k, kind=kind)
    fused, unfused = _fused_and_unfused(S, di, k, W, relu, qi, ki)
    lens = np.arange(1, S + 1)
    check_rows_ascending(fused, lens, k)
    # the same fp32 scores: the fused selection equals the stored-score one
    assert np.array_equal(fused, unfused)
    rows = np.unique(np.linspace(0, S - 1, min(S, 64)).round().astype(int))
    Y = oracle.index_scores(qi, ki, rows=rows, relu=bool(relu))
    ref = oracle.topk(Y, rows + 1, k, W)
    for i, t in enumerate(rows):
        compare_support(fused[t], ref[i], Y[i], t + 1, k, W)


def test_indexer_topk_fused_headline_sampled():
    S, di, k = 32768, 128, 2048
    say(f"fused indexer top-k S={S} k={k}")
    inp = make_inputs(S, 32, 8, 128, index_dim=di, dtype="bf16", needles=128, seed=4)
    fused, unfused = _fused_and_unfused(S, di, k, 0, 1, inp.q_idx, inp.k_idx)
    assert np.array_equal(fused, unfused)
    rows = np.array([0, 2046, 2047, 2048, 4095, 4096, 20000, 32767])
    Y = oracle.index_scores(inp.q_idx, inp.k_idx, rows=rows)
    ref = oracle.topk(Y, rows + 1, k)
    for i, t in enumerate(rows):
        compare_support(fused[t], ref[i], Y[i], t + 1, k)


# ------------------------------------------------- per-KV-group supports (f3)
from synth import make_support  # noqa: E402
from helpers import check_attention, max_err  # noqa: E402


@pytest.mark.parametrize("S,Hq,Hkv,d,b,dtype", [(200, 8, 2, 64, 1, "f32"),
                                                (300, 8, 2, 128, 16, "bf16"),
                                                (257, 12, 3, 64, 4, "bf16")])
def test_group_mass_and_topk(S, Hq, Hkv, d, b, dtype):
    say(f"per-group mass+topk S={S} Hq={Hq} Hkv={Hkv} d={d} b={b} {dtype}")
    k = 24
    inp = make_inputs(S, Hq, Hkv, d, dtype=dtype, seed=S + b, peaked=True, needles=4)
    p = B.Problem(S, Hq, Hkv, d, topk=k, block_q=b, dtype=dtype, head_axis=1, local_window=2)
    q, kk, v = inp.q.cuda(), inp.k.cuda(), inp.v.cuda()
    lse = torch.empty(S, Hq, device="cuda")
    B.sp_dense_attn(p, q, kk, v, None, lse)
    R = p.num_blocks
    mass = torch.full((Hkv, R, S), float("nan"), device="cuda")
    B.sp_oracle_support(p, q, kk, lse, mass)
    idx = torch.empty(Hkv, R, k, dtype=torch.int32, device="cuda")
    B.sp_topk_select(p, mass, idx)
    torch.cuda.synchronize()
    got, gidx = mass.cpu().double().numpy(), idx.cpu().numpy()
    lens = np.array([min(r * b + b, S) for r in range(R)])
    for j in range(Hkv):
        ref = oracle.support_scores("oracle", range(R), b, q=inp.q, k=inp.k, group=j)
        ref_idx = oracle.topk(ref, lens, k, 2)
        check_rows_ascending(gidx[j], lens, k)
        for r in range(R):
            L = lens[r]
            assert max_err(got[j, r, :L], ref[r, :L]) <= 1e-4 * np.abs(ref[r, :L]).max()
            assert np.all(np.isnan(got[j, r, L:]))
            compare_support(gidx[j, r], ref_idx[r], ref[r], L, k, 2)


@pytest.mark.parametrize("S,Hq,Hkv,d,b,dtype", [(300, 8, 2, 128, 64, "bf16"),
                                                (300, 8, 2, 64, 16, "bf16"),
                                                (257, 8, 4, 128, 1, "bf16"),
                                                (200, 6, 3, 64, 3, "bf16"),
                                                (150, 4, 2, 64, 8, "f32")])
def test_group_sparse_attention(S, Hq, Hkv, d, b, dtype):
    say(f"per-group sparse S={S} Hq={Hq} Hkv={Hkv} d={d} b={b} {dtype}")
    k = 40
    inp = make_inputs(S, Hq, Hkv, d, dtype=dtype, seed=S + d, peaked=True)
    tables = torch.stack([make_support(S, b, k, seed=10 + j, shuffle=j % 2 == 1)
                          for j in range(Hkv)])
    p = B.Problem(S, Hq, Hkv, d, topk=k, block_q=b, dtype=dtype, head_axis=1)
    o = torch.empty(S, Hq, d, dtype=inp.q.dtype, device="cuda")
    B.sp_sparse_gqa_attn(p, inp.q.cuda(), inp.k.cuda(), inp.v.cuda(), tables.cuda(), o)
    torch.cuda.synchronize()
    ref = oracle.sparse(inp.q, inp.k, inp.v, tables, b)
    ref_abs = oracle.sparse(inp.q, inp.k, inp.v.abs(), tables, b)
    check_attention(o.cpu().double().numpy(), ref, ref_abs, dtype)


def test_indexer_rejects_per_group_supports():
    p = B.Problem(64, 8, 2, 64, index_dim=64, topk=8, head_axis=1)
    x = torch.zeros(64, 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.SparsePrefillError):
        B.sp_indexer_scores(p, x, x, torch.empty(64, 64, device="cuda"))


# ------------------------------------------------------- paged K/V cache (f3)
def _paged(k, v, ps, seed, extra=3):
    """Scatter contiguous K/V over a larger cache of pages through a random table."""
    S = k.shape[0]
    npg = (S + ps - 1) // ps
    perm = np.random.default_rng(seed).permutation(npg + extra)[:npg].astype(np.int32)
    kp = torch.zeros((npg + extra, ps) + tuple(k.shape[1:]), dtype=k.dtype)
    vp = torch.zeros_like(kp)
    for lp in range(npg):
        n = min(ps, S - lp * ps)
        kp[perm[lp], :n] = k[lp * ps: lp * ps + n]
        vp[perm[lp], :n] = v[lp * ps: lp * ps + n]
    return kp, vp, torch.from_numpy(perm)


@pytest.mark.parametrize("S,Hq,Hkv,d,b,dtype,ps,head_axis", [
    (300, 8, 2, 128, 64, "bf16", 16, 0),
    (300, 8, 2, 256, 16, "bf16", 16, 1),
    (300, 8, 2, 64, 16, "bf16", 7, 1),
    (257, 8, 4, 128, 1, "bf16", 32, 0),
    (200, 6, 3, 64, 4, "bf16", 1, 1),
    (150, 4, 2, 64, 8, "f32", 10, 0),
])
def test_paged_sparse_attention(S, Hq, Hkv, d, b, dtype, ps, head_axis):
    say(f"paged sparse S={S} d={d} b={b} {dtype} page={ps} head_axis={head_axis}")
    k_ = 40
    inp = make_inputs(S, Hq, Hkv, d, dtype=dtype, seed=S + ps, peaked=True)
    if head_axis:
        table = torch.stack([make_support(S, b, k_, seed=30 + j) for j in range(Hkv)])
    else:
        table = make_support(S, b, k_, seed=30, shuffle=True)
    kp, vp, pt = _paged(inp.k, inp.v, ps, seed=S)
    p = B.Problem(S, Hq, Hkv, d, topk=k_, block_q=b, dtype=dtype, head_axis=head_axis)
    o = torch.empty(S, Hq, d, dtype=inp.q.dtype, device="cuda")
    B.sp_sparse_gqa_attn_paged(p, inp.q.cuda(), kp.cuda(), vp.cuda(), pt.cuda(), table.cuda(), o)
    # a logical page outside the cache drops its positions
    bad = pt.clone()
    bad[1] = kp.shape[0] + 5
    o_bad = torch.empty_like(o)
    B.sp_sparse_gqa_attn_paged(p, inp.q.cuda(), kp.cuda(), vp.cuda(), bad.cuda(), table.cuda(),
                               o_bad)
    torch.cuda.synchronize()
    ref = oracle.sparse_paged(inp.q, kp, vp, pt, table, b)
    ref_abs = oracle.sparse_paged(inp.q, kp, vp.abs(), pt, table, b)
    check_attention(o.cpu().double().numpy(), ref, ref_abs, dtype)
    ref_bad = oracle.sparse_paged(inp.q, kp, vp, bad, table, b)
    ref_bad_abs = oracle.sparse_paged(inp.q, kp, vp.abs(), bad, table, b)
    check_attention(o_bad.cpu().double().numpy(), ref_bad, ref_bad_abs, dtype)
    # the paged result is the contiguous one
    o_c = torch.empty_like(o)
    B.sp_sparse_gqa_attn(p, inp.q.cuda(), inp.k.cuda(), inp.v.cuda(), table.cuda(), o_c)
    torch.cuda.synchronize()
    assert torch.equal(o, o_c)


@pytest.mark.parametrize("k_", [2048, 2049])
def test_paged_head_dim_256_long_support(k_):
    """At head_dim 256 the paged block kernel caches supports of up to 2048
    entries (its K/V tiles fill most of LDS); a longer support takes the
    row-wise kernel. Both match the contiguous call, which is held to the
    oracle on sampled rows of sharp inputs (32 key tiles, rescale after the
    first)."""
    S, Hq, Hkv, d, b = 2300, 8, 2, 256, 64
    say(f"paged d=256 k={k_}")
    inp = make_inputs(S, Hq, Hkv, d, dtype="bf16", seed=k_, peaked=True, unit_v=True,
                      k_ramp=8.0)
    table = make_support(S, b, k_, seed=7, shuffle=True)
    kp, vp, pt = _paged(inp.k, inp.v, 64, seed=S)
    p = B.Problem(S, Hq, Hkv, d, topk=k_, block_q=b, dtype="bf16")
    o = torch.empty(S, Hq, d, dtype=inp.q.dtype, device="cuda")
    B.sp_sparse_gqa_attn_paged(p, inp.q.cuda(), kp.cuda(), vp.cuda(), pt.cuda(), table.cuda(), o)
    o_c = torch.empty_like(o)
    B.sp_sparse_gqa_attn(p, inp.q.cuda(), inp.k.cuda(), inp.v.cuda(), table.cuda(), o_c)
    torch.cuda.synchronize()
    rows = np.concatenate([np.arange(r * b, min(r * b + b, S), 9) for r in (0, 17, 33, 35)])
    ref = oracle.sparse(inp.q, inp.k, inp.v, table, b, rows=rows)
    ref_abs = oracle.sparse(inp.q, inp.k, inp.v.abs(), table, b, rows=rows)
    check_attention(o_c.cpu().double().numpy()[rows], ref, ref_abs, "bf16", "contiguous: ")
    if k_ <= 2048:
        assert torch.equal(o, o_c)
    else:   # row-wise (paged) against the block kernel (contiguous)
        check_attention(o.cpu().double().numpy()[rows], ref, ref_abs, "bf16", "paged: ")


# ------------------------------------------------ chunked prefill rows (f3)
from synth import make_scores  # noqa: E402


@pytest.mark.parametrize("S,qo,b,d,dtype", [(300, 128, 64, 128, "bf16"), (300, 48, 16, 64, "bf16"),
                                            (257, 77, 1, 128, "bf16"), (200, 40, 4, 64, "f32"),
                                            (200, 199, 1, 64, "bf16")])
def test_chunked_sparse_attention(S, qo, b, d, dtype):
    say(f"chunked sparse S={S} q_offset={qo} b={b} d={d} {dtype}")
    Hq, Hkv, k = 8, 2, 40
    inp = make_inputs(S, Hq, Hkv, d, dtype=dtype, seed=S + qo, peaked=True)
    full = make_support(S, b, k, seed=qo)            # tables of the whole sequence
    table = full[qo // b:].contiguous()              # the chunk's blocks
    p = B.Problem(S, Hq, Hkv, d, topk=k, block_q=b, dtype=dtype, q_offset=qo)
    o = torch.empty(S - qo, Hq, d, dtype=inp.q.dtype, device="cuda")
    B.sp_sparse_gqa_attn(p, inp.q[qo:].contiguous().cuda(), inp.k.cuda(), inp.v.cuda(),
                         table.cuda(), o)
    kp, vp, pt = _paged(inp.k, inp.v, 16, seed=S)
    o2 = torch.empty_like(o)
    B.sp_sparse_gqa_attn_paged(p, inp.q[qo:].contiguous().cuda(), kp.cuda(), vp.cuda(),
                               pt.cuda(), table.cuda(), o2)
    torch.cuda.synchronize()
    ref = oracle.sparse(inp.q, inp.k, inp.v, full, b, rows=np.arange(qo, S))
    ref_abs = oracle.sparse(inp.q, inp.k, inp.v.abs(), full, b, rows=np.arange(qo, S))
    check_attention(o.cpu().double().numpy(), ref, ref_abs, dtype)
    assert torch.equal(o, o2)


@pytest.mark.parametrize("S,qo,b,W", [(300, 100, 1, 0), (300, 96, 32, 5), (5000, 4096, 64, 0)])
def test_chunked_topk(S, qo, b, W):
    say(f"chunked topk S={S} q_offset={qo} b={b} W={W}")
    k = 37
    R = (S - qo + b - 1) // b
    scores = make_scores(R, S, seed=S + qo, kind="relu")
    p = B.Problem(S, 1, 1, 64, topk=k, block_q=b, local_window=W, dtype="f32", q_offset=qo)
    idx = torch.empty(R, k, dtype=torch.int32, device="cuda")
    B.sp_topk_select(p, scores.cuda(), idx)
    torch.cuda.synchronize()
    lens = np.array([min(qo + r * b + b, S) for r in range(R)])
    ref = oracle.topk(scores.numpy().astype(np.float64), lens, k, W)
    assert np.array_equal(idx.cpu().numpy(), ref)


@pytest.mark.parametrize("S,qo,b,di", [(700, 100, 1, 128), (1200, 512, 64, 128),
                                       (700, 128, 64, 64), (700, 64, 16, 256)])
def test_chunked_indexer_scores(S, qo, b, di):
    say(f"chunked indexer S={S} q_offset={qo} b={b} d_idx={di}")
    inp = make_inputs(S, 1, 1, 64, index_dim=di, dtype="bf16", seed=S + b, needles=4)
    p = B.Problem(S, 1, 1, 64, index_dim=di, topk=8, block_q=b, q_offset=qo)
    R = p.num_blocks
    sc = torch.full((R, S), float("nan"), device="cuda")
    B.sp_indexer_scores(p, inp.q_idx[qo:].contiguous().cuda(), inp.k_idx.cuda(), sc)
    torch.cuda.synchronize()
    units = range(qo // b, qo // b + R)
    ref = oracle.support_scores("indexer", units, b, q_idx=inp.q_idx, k_idx=inp.k_idx)
    got = sc.cpu().double().numpy()
    scale = np.abs(ref).max()
    for r in range(R):
        L = min(qo + r * b + b, S)
        assert max_err(got[r, :L], ref[r, :L]) <= 2e-6 * scale
        assert np.all(np.isnan(got[r, L:]))


def test_chunked_dense_and_pipeline_equal_whole_sequence():
    S, Hq, Hkv, d, di, k, b, qo = 640, 8, 2, 128, 128, 64, 64, 512
    say(f"chunked pipeline S={S} chunks [0,{qo}) [{qo},{S})")
    inp = make_inputs(S, Hq, Hkv, d, index_dim=di, dtype="bf16", seed=7, needles=8)
    dev = inp.to("cuda")

    def run(p, q, qi, S_):
        R = p.num_blocks
        sc = torch.empty(R, S_, device="cuda")
        B.sp_indexer_scores(p, qi, dev.k_idx[:S_].contiguous(), sc)
        idx = torch.empty(R, k, dtype=torch.int32, device="cuda")
        B.sp_topk_select(p, sc, idx)
        o = torch.empty(p.num_queries, Hq, d, dtype=torch.bfloat16, device="cuda")
        B.sp_sparse_gqa_attn(p, q, dev.k[:S_].contiguous(), dev.v[:S_].contiguous(), idx, o)
        return idx, o

    whole = B.Problem(S, Hq, Hkv, d, index_dim=di, topk=k, block_q=b)
    idx_w, o_w = run(whole, dev.q, dev.q_idx, S)
    first = B.Problem(qo, Hq, Hkv, d, index_dim=di, topk=k, block_q=b)
    idx_1, o_1 = run(first, dev.q[:qo].contiguous(), dev.q_idx[:qo].contiguous(), qo)
    second = B.Problem(S, Hq, Hkv, d, index_dim=di, topk=k, block_q=b, q_offset=qo)
    idx_2, o_2 = run(second, dev.q[qo:].contiguous(), dev.q_idx[qo:].contiguous(), S)
    lse = torch.empty(S - qo, Hq, device="cuda")
    o_d = torch.empty(S - qo, Hq, d, dtype=torch.bfloat16, device="cuda")
    B.sp_dense_attn(second, dev.q[qo:].contiguous(), dev.k, dev.v, o_d, lse)
    torch.cuda.synchronize()
    # the same scores and selections, chunk by chunk
    assert torch.equal(torch.cat([idx_1, idx_2]), idx_w)
    # a block's output depends only on its support and its own rows
    assert torch.equal(torch.cat([o_1, o_2]), o_w)
    ref_o, ref_lse = oracle.dense(inp.q, inp.k, inp.v, rows=np.arange(qo, S))
    ref_abs, _ = oracle.dense(inp.q, inp.k, inp.v.abs(), rows=np.arange(qo, S))
    check_attention(o_d.cpu().double().numpy(), ref_o, ref_abs, "bf16")
    assert max_err(lse.cpu().double().numpy(), ref_lse) <= 1e-4


# ------------------------------------------------------ d = d_idx = 256 (f3)
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_head_dim_256(dtype):
    S, Hq, Hkv, d, b, k = 200, 8, 2, 256, 16, 48
    say(f"head_dim 256 {dtype}")
    inp = make_inputs(S, Hq, Hkv, d, index_dim=256, dtype=dtype, seed=256, peaked=True,
                      needles=4)
    dev = inp.to("cuda")
    p = B.Problem(S, Hq, Hkv, d, index_dim=256, topk=k, block_q=b, dtype=dtype)
    o = torch.empty(S, Hq, d, dtype=inp.q.dtype, device="cuda")
    lse = torch.empty(S, Hq, device="cuda")
    B.sp_dense_attn(p, dev.q, dev.k, dev.v, o, lse)
    mass = torch.full((p.num_blocks, S), float("nan"), device="cuda")
    B.sp_oracle_support(p, dev.q, dev.k, lse, mass)
    table = make_support(S, b, k, seed=3)
    o_s = torch.empty_like(o)
    B.sp_sparse_gqa_attn(p, dev.q, dev.k, dev.v, table.cuda(), o_s)
    p1 = B.Problem(S, Hq, Hkv, d, index_dim=256, topk=k, block_q=1, dtype=dtype)
    t1 = make_support(S, 1, k, seed=4)
    o_q = torch.empty_like(o)
    B.sp_sparse_gqa_attn(p1, dev.q, dev.k, dev.v, t1.cuda(), o_q)
    torch.cuda.synchronize()
    ref_o, ref_lse = oracle.dense(inp.q, inp.k, inp.v)
    ref_abs, _ = oracle.dense(inp.q, inp.k, inp.v.abs())
    check_attention(o.cpu().double().numpy(), ref_o, ref_abs, dtype, "dense: ")
    assert max_err(lse.cpu().double().numpy(), ref_lse) <= (1e-5 if dtype == "f32" else 1e-4)
    ref_m = oracle.support_scores("oracle", range(p.num_blocks), b, q=inp.q, k=inp.k)
    got_m = mass.cpu().double().numpy()
    for r in range(p.num_blocks):
        L = min(r * b + b, S)
        assert max_err(got_m[r, :L], ref_m[r, :L]) <= 1e-4 * np.abs(ref_m[r, :L]).max()
    check_attention(o_s.cpu().double().numpy(), oracle.sparse(inp.q, inp.k, inp.v, table, b),
                    oracle.sparse(inp.q, inp.k, inp.v.abs(), table, b), dtype, "block: ")
    check_attention(o_q.cpu().double().numpy(), oracle.sparse(inp.q, inp.k, inp.v, t1, 1),
                    oracle.sparse(inp.q, inp.k, inp.v.abs(), t1, 1), dtype, "per query: ")

"""Pins for the fp64 CPU oracle, each tied to something other than the oracle.

Pins used: torch's scaled_dot_product_attention (an independent library
routine) for dense and restricted attention and, through one-hot values, for
the attention weights behind the head-averaged mass; torch matmul for the
indexer contraction; closed forms (zero queries, constant values, the
causal-pair count); invariants the paper states (mass rows sum to one,
restricted weights sum to one, each query masks a shared support causally,
full budget equals dense); brute-force enumeration of k-subsets for top-k;
and the sparsities the paper prints (tests/golden/causal_sparsity.txt).
"""
import itertools
import os

import numpy as np
import pytest
import torch

import oracle
from synth import make_inputs, make_scores, make_support

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F = torch.nn.functional


def _bhsd(x):
    return torch.as_tensor(np.asarray(x, dtype=np.float64)).permute(1, 0, 2)[None]


def sdpa_causal(q, k, v):
    out = F.scaled_dot_product_attention(_bhsd(q), _bhsd(k), _bhsd(v), is_causal=True,
                                         enable_gqa=True)
    return out[0].permute(1, 0, 2).numpy()


def sdpa_masked(q, k, v, mask):
    m = torch.as_tensor(mask)[None, None]
    out = F.scaled_dot_product_attention(_bhsd(q), _bhsd(k), _bhsd(v), attn_mask=m,
                                         enable_gqa=True)
    return out[0].permute(1, 0, 2).numpy()


def f64(t):
    return t.to(torch.float64).numpy()


SHAPES = [(1, 1), (4, 4), (4, 2), (4, 1), (8, 2)]


# ------------------------------------------------------------------ dense
@pytest.mark.parametrize("S", [1, 2, 7, 64, 130])
@pytest.mark.parametrize("heads", SHAPES)
@pytest.mark.parametrize("d", [8, 64])
def test_dense_matches_sdpa(S, heads, d):
    Hq, Hkv = heads
    inp = make_inputs(S, Hq, Hkv, d, dtype="f32", needles=min(2, S), seed=11 + S, peaked=True)
    o, lse = oracle.dense(inp.q, inp.k, inp.v)
    ref = sdpa_causal(f64(inp.q), f64(inp.k), f64(inp.v))
    assert np.abs(o - ref).max() < 1e-12
    # normaliser against torch.logsumexp of causally masked logits
    q, k = torch.as_tensor(f64(inp.q)), torch.as_tensor(f64(inp.k))
    kk = k.repeat_interleave(Hq // Hkv, dim=1)
    logits = torch.matmul(q.permute(1, 0, 2), kk.permute(1, 2, 0).contiguous()) / np.sqrt(d)
    causal = torch.ones(S, S, dtype=torch.bool).tril()
    ref_lse = torch.logsumexp(logits.masked_fill(~causal, -float("inf")), dim=-1).T.numpy()
    assert np.abs(lse - ref_lse).max() < 1e-12


def test_dense_closed_forms():
    S, Hq, Hkv, d = 40, 4, 2, 16
    inp = make_inputs(S, Hq, Hkv, d, dtype="f32", seed=5)
    q0 = np.zeros((S, Hq, d))
    v = f64(inp.v)
    o, lse = oracle.dense(q0, f64(inp.k), v)
    t = np.arange(S)
    # zero queries: uniform weights, lse = log(t+1), o_t = mean(v_0..v_t)
    assert np.abs(lse - np.log(t + 1)[:, None]).max() < 1e-13
    cm = np.cumsum(v, axis=0) / (t + 1)[:, None, None]
    assert np.abs(o - np.repeat(cm, Hq // Hkv, axis=1)).max() < 1e-13
    # t = 0 attends only to key 0
    o, _ = oracle.dense(f64(inp.q), f64(inp.k), v, rows=[0])
    assert np.array_equal(o[0], np.repeat(v[0], Hq // Hkv, axis=0))


# ------------------------------------------------------------------- mass
@pytest.mark.parametrize("heads", SHAPES)
def test_mass_is_head_average_of_attention_weights(heads):
    Hq, Hkv = heads
    S, d = 37, 8
    inp = make_inputs(S, Hq, Hkv, d, dtype="f32", seed=21, peaked=True)
    P = oracle.mass(inp.q, inp.k)
    # attention weights from the library: values = identity gives o[t] = A[t, :]
    eye = np.broadcast_to(np.eye(S)[:, None, :], (S, Hkv, S)).copy()
    A = sdpa_causal(f64(inp.q), f64(inp.k), eye)          # [S, Hq, S]
    assert np.abs(P - A.mean(axis=1)).max() < 1e-13
    assert np.abs(P.sum(axis=1) - 1.0).max() < 1e-13     # each row sums to one
    assert np.all(P[np.triu_indices(S, 1)] == 0.0)


# ---------------------------------------------------------------- indexer
@pytest.mark.parametrize("relu", [True, False])
def test_index_scores_match_matmul(relu):
    S, di = 50, 16
    inp = make_inputs(S, 1, 1, 8, index_dim=di, dtype="f32", seed=31)
    Z = oracle.index_scores(inp.q_idx, inp.k_idx, relu=relu)
    qi, ki = torch.as_tensor(f64(inp.q_idx)), torch.as_tensor(f64(inp.k_idx))
    ref = (qi @ ki.T / np.sqrt(di)).numpy()
    if relu:
        ref = np.maximum(ref, 0.0)
    ref = np.tril(ref)
    assert np.abs(Z - ref).max() < 1e-13


# -------------------------------------------------------------- aggregate
def test_aggregate_rules():
    rng = np.random.default_rng(0)
    S = 20
    trows = np.arange(8, 14)
    X = rng.standard_normal((len(trows), S))
    garbage = X.copy()
    for i, t in enumerate(trows):
        garbage[i, t + 1:] = 1e9       # non-causal entries must be ignored
    Ymax = oracle.aggregate(garbage, trows, "max")
    Ysum = oracle.aggregate(garbage, trows, "sum")
    for s in range(S):
        members = [X[i, s] for i, t in enumerate(trows) if t >= s]
        if not members:
            assert Ymax[s] == 0 and Ysum[s] == 0
            continue
        assert Ymax[s] == max(members) and Ymax[s] in members
        assert abs(Ysum[s] - sum(members)) < 1e-12
    # constant rows: SUM counts the queries of the block at or after s
    ones = np.ones((len(trows), S))
    cnt = oracle.aggregate(ones, trows, "sum")
    assert np.array_equal(cnt[:14], np.array([min(6, 13 - s + 1) for s in range(14)], float))
    # one query: identity on the causal prefix
    assert np.array_equal(oracle.aggregate(X[:1], trows[:1], "max")[:9], X[0, :9])


# ------------------------------------------------------------------- top-k
def _dominates(a, b, y):
    return y[a] > y[b] or (y[a] == y[b] and a < b)


@pytest.mark.parametrize("seed", range(6))
def test_topk_brute_force_subsets(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(5, 10))
    k = int(rng.integers(1, L))
    W = int(rng.integers(0, k + 1)) if seed % 2 else 0
    y = rng.integers(0, 3, size=L).astype(np.float64)   # many exact ties
    out = oracle.topk(y, [L], k, W)[0]
    Wf = min(W, k)
    forced = set(range(L - Wf, L))
    cands = list(range(L - Wf))
    winners = []
    for sub in itertools.combinations(cands, k - Wf):
        rest = [b for b in cands if b not in sub]
        if all(_dominates(a, b, y) for a in sub for b in rest):
            winners.append(set(sub))
    assert len(winners) == 1
    expect = sorted(winners[0] | forced)
    assert list(out) == expect


@pytest.mark.parametrize("kind", ["gauss", "relu", "coarse", "const"])
def test_topk_matches_lexsort(kind):
    Y = make_scores(12, 300, seed=7, kind=kind).numpy().astype(np.float64)
    lens = np.array([1, 5, 40, 41, 100, 200, 257, 299, 300, 300, 64, 65])
    k, W = 40, 8
    out = oracle.topk(Y, lens, k, W)
    for i, L in enumerate(lens):
        if L <= k:
            expect = list(range(L)) + [-1] * (k - L)
        else:
            c = np.arange(L - W)
            order = np.lexsort((c, -Y[i, : L - W]))
            expect = sorted(list(c[order[: k - W]]) + list(range(L - W, L)))
        assert list(out[i]) == expect


def test_topk_k1_is_first_argmax():
    Y = make_scores(20, 64, seed=3, kind="coarse").numpy().astype(np.float64)
    out = oracle.topk(Y, np.full(20, 64), 1, 0)
    assert np.array_equal(out[:, 0], np.argmax(Y, axis=1))


def test_kept_pairs_closed_form_and_printed_sparsity():
    S, k = 300, 37
    Y = make_scores(S, S, seed=1).numpy().astype(np.float64)
    out = oracle.topk(Y, np.arange(1, S + 1), k)
    kept = int((out >= 0).sum())
    assert np.array_equal((out >= 0).sum(axis=1), np.minimum(np.arange(1, S + 1), k))
    assert kept == k * S - k * (k - 1) // 2
    rows = [ln.split() for ln in open(os.path.join(GOLDEN, "causal_sparsity.txt"))
            if ln.strip() and not ln.startswith("#")]
    assert len(rows) == 9
    for r in rows:
        S, k, pct, dec = int(r[0]), int(r[1]), float(r[2]), int(r[3])
        kept = k * S - k * (k - 1) // 2
        sparsity = 100.0 * (1.0 - kept / (S * (S + 1) / 2))
        assert round(sparsity, dec) == pytest.approx(pct), (S, k, sparsity)


# ------------------------------------------------------------------ sparse
@pytest.mark.parametrize("heads", SHAPES)
@pytest.mark.parametrize("b", [1, 3, 4, 37, 38])
def test_sparse_matches_masked_sdpa(heads, b):
    Hq, Hkv = heads
    S, d, kk = 37, 8, 9
    inp = make_inputs(S, Hq, Hkv, d, dtype="f32", seed=41, peaked=True)
    idx = make_support(S, b, kk, seed=b).numpy()
    o = oracle.sparse(inp.q, inp.k, inp.v, idx, b)
    mask = np.zeros((S, S), dtype=bool)
    for t in range(S):
        for s in idx[t // b]:
            if 0 <= s <= t:
                mask[t, s] = True
    nonempty = mask.any(axis=1)
    ref = sdpa_masked(f64(inp.q), f64(inp.k), f64(inp.v), mask)
    assert np.abs(o[nonempty] - ref[nonempty]).max() < 1e-12
    assert np.all(o[~nonempty] == 0.0)


@pytest.mark.parametrize("b", [1, 5, 64])
def test_sparse_full_budget_is_dense(b):
    S, Hq, Hkv, d = 64, 4, 2, 16
    inp = make_inputs(S, Hq, Hkv, d, dtype="f32", seed=2, peaked=True)
    R = (S + b - 1) // b
    idx = np.tile(np.arange(S, dtype=np.int32), (R, 1))
    o = oracle.sparse(inp.q, inp.k, inp.v, idx, b)
    assert np.abs(o - sdpa_causal(f64(inp.q), f64(inp.k), f64(inp.v))).max() < 1e-12


def test_sparse_invariances_and_unit_weights():
    S, Hq, Hkv, d, b, kk = 50, 4, 2, 8, 4, 12
    inp = make_inputs(S, Hq, Hkv, d, dtype="f32", seed=9, peaked=True)
    idx = make_support(S, b, kk, seed=1).numpy()
    o = oracle.sparse(inp.q, inp.k, inp.v, idx, b)
    rng = np.random.default_rng(0)
    perm = np.stack([rng.permutation(r) for r in idx])
    padded = np.concatenate([perm, np.full((idx.shape[0], 5), -1, np.int32)], axis=1)
    o2 = oracle.sparse(inp.q, inp.k, inp.v, padded, b)
    assert np.abs(o - o2).max() < 1e-14
    ones = np.ones((S, Hkv, d))
    o1 = oracle.sparse(inp.q, inp.k, ones, idx, b)
    nonempty = np.abs(o1).sum(axis=(1, 2)) > 0
    assert np.abs(o1[nonempty] - 1.0).max() < 1e-14   # weights sum to one


def test_sparse_empty_support_is_zero():
    S, b = 8, 4
    inp = make_inputs(S, 2, 1, 8, dtype="f32", seed=3)
    idx = np.array([[2], [6]], dtype=np.int32)   # k=1 < b: queries 4,5 see nothing
    o = oracle.sparse(inp.q, inp.k, inp.v, idx, b, rows=[0, 1, 4, 5, 6, 7])
    assert np.all(o[0] == 0) and np.all(o[1] == 0) and np.all(o[2] == 0) and np.all(o[3] == 0)
    v = f64(inp.v)
    assert np.allclose(o[4], v[6, 0][None]) and np.allclose(o[5], v[6, 0][None])


# --------------------------------------------------------------- pipelines
def test_single_head_oracle_support_is_topk_of_logits():
    S, d, k = 96, 16, 10
    inp = make_inputs(S, 1, 1, d, dtype="f32", seed=4, peaked=True)
    Y = oracle.support_scores("oracle", range(S), 1, q=inp.q, k=inp.k)
    idx = oracle.select(Y, range(S), 1, S, k)
    q, kk = torch.as_tensor(f64(inp.q))[:, 0], torch.as_tensor(f64(inp.k))[:, 0]
    logits = (q @ kk.T).numpy()
    for t in range(S):
        if t + 1 <= k:
            assert list(idx[t][: t + 1]) == list(range(t + 1))
            continue
        order = np.lexsort((np.arange(t + 1), -logits[t, : t + 1]))
        assert list(idx[t]) == sorted(order[:k])


def test_support_contains_top_mass_tokens():
    S, k = 200, 16
    inp = make_inputs(S, 4, 2, 16, dtype="f32", seed=8, peaked=True)
    P = oracle.mass(inp.q, inp.k)
    idx = oracle.topk(P, np.arange(1, S + 1), k)
    for t in range(k, S):
        sel = set(idx[t])
        thr = np.sort(P[t, : t + 1])[::-1][k]        # (k+1)-th largest mass
        assert all(s in sel for s in np.nonzero(P[t, : t + 1] > thr)[0])
        assert int(np.argmax(P[t, : t + 1])) in sel


def test_block_support_masks_each_query_causally():
    # a query early in a block must not see support entries beyond itself
    S, b, k = 16, 8, 16
    inp = make_inputs(S, 2, 1, 8, dtype="f32", seed=6, peaked=True)
    idx = oracle.select(oracle.support_scores("oracle", [0, 1], b, q=inp.q, k=inp.k),
                        [0, 1], b, S, k)
    assert list(idx[0][:8]) == list(range(8)) and list(idx[1]) == list(range(16))
    o = oracle.sparse(inp.q, inp.k, inp.v, idx, b)
    ref = sdpa_causal(f64(inp.q), f64(inp.k), f64(inp.v))
    assert np.abs(o - ref).max() < 1e-12


def test_needles_retrieved_indexer_mode():
    S, k = 1024, 128
    inp = make_inputs(S, 4, 2, 64, index_dim=64, dtype="bf16", needles=16, seed=2)
    units = sorted(set(inp.probe_query.tolist()))
    Y = oracle.support_scores("indexer", units, 1, q_idx=inp.q_idx, k_idx=inp.k_idx)
    idx = oracle.select(Y, units, 1, S, k)
    sup = {u: set(r) for u, r in zip(units, idx)}
    for p, r in zip(inp.needle_pos, inp.probe_query):
        assert p in sup[int(r)]


def test_needles_retrieved_oracle_mode_tiny_config():
    from synth import get_workload
    w = get_workload("oracle_tiny_512")
    inp = make_inputs(w.seq_len, w.num_q_heads, w.num_kv_heads, w.head_dim, dtype=w.dtype,
                      needles=w.needles, seed=w.seed)
    units = sorted(set(inp.probe_query.tolist()))
    Y = oracle.support_scores("oracle", units, 1, q=inp.q, k=inp.k)
    idx = oracle.select(Y, units, 1, w.seq_len, w.topk)
    sup = {u: set(r) for u, r in zip(units, idx)}
    for p, r in zip(inp.needle_pos, inp.probe_query):
        assert p in sup[int(r)]

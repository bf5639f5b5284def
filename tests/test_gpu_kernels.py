"""GPU parity, one entry point at a time, against the fp64 oracle.

Inputs come from the seeded generator only (supports and score rows too), so
each kernel is checked in isolation from the others. Sizes span several
tiles and end in ragged tails.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_07703_amd import binding as B
from synth import make_inputs, make_scores, make_support

from helpers import (check_attention, check_rows_ascending, cuda, f64, logit_rise, max_err,
                     say)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()


def _inp(S, Hq, Hkv, d, di=0, dtype="bf16", seed=0, peaked=False, needles=0):
    return make_inputs(S, Hq, Hkv, d, index_dim=di, dtype=dtype, needles=needles, seed=seed,
                       peaked=peaked)


# ------------------------------------------------------------ sparse attention
def ref_sparse(inp, idx, b, rows=None):
    """Oracle outputs and the same attention over |V| (the scale of the bound)."""
    return (oracle.sparse(inp.q, inp.k, inp.v, idx, b, rows=rows),
            oracle.sparse(inp.q, inp.k, inp.v.abs(), idx, b, rows=rows))


SPARSE_CASES = [
    # S, Hq, Hkv, d, dtype, b, k
    (1, 4, 2, 64, "f32", 1, 1),
    (300, 4, 2, 64, "f32", 1, 37),
    (300, 6, 2, 64, "f32", 16, 64),
    (300, 4, 4, 128, "f32", 64, 100),
    (257, 8, 2, 128, "bf16", 1, 64),
    (257, 8, 2, 128, "bf16", 64, 128),
    (300, 16, 4, 128, "bf16", 16, 200),
    (300, 2, 1, 64, "bf16", 7, 5),
    (200, 8, 8, 128, "bf16", 1, 250),
    (520, 32, 8, 128, "bf16", 64, 256),
    (520, 32, 8, 128, "bf16", 128, 96),
    (300, 32, 2, 64, "bf16", 1, 100),      # G = 16: every MFMA column a head
    (400, 12, 4, 128, "bf16", 1, 33),      # G = 3, ragged last tile
    (260, 4, 1, 64, "bf16", 3, 2100),      # support row longer than one LDS chunk
    (260, 8, 2, 256, "bf16", 1, 2100),     # the same at d = 256
    (130, 34, 2, 64, "bf16", 1, 40),       # G = 17: row-wise path
]


@pytest.mark.parametrize("case", SPARSE_CASES, ids=lambda c: "-".join(map(str, c)))
def test_sparse_attention(case):
    S, Hq, Hkv, d, dtype, b, k = case
    say(f"sparse {case}")
    inp = _inp(S, Hq, Hkv, d, dtype=dtype, seed=S + k, peaked=(dtype == "f32"))
    idx = make_support(S, b, k, seed=b)
    p = B.Problem(S, Hq, Hkv, d, topk=k, block_q=b, dtype=dtype)
    o = torch.empty(S, Hq, d, dtype=inp.q.dtype, device="cuda")
    B.sp_sparse_gqa_attn(p, cuda(inp.q), cuda(inp.k), cuda(inp.v), cuda(idx), o)
    torch.cuda.synchronize()
    check_attention(f64(o), *ref_sparse(inp, idx, b), dtype)


# Multi-tile supports with sharp attention: unscaled Q and K (logits of unit
# spread), key rows ramped so later tiles carry larger logits (the running
# maximum rises by more than 8 in base 2 after the first tile: the rescale
# path), V of unit spread; some tables shuffled so rises land at random tiles.
SHARP_CASES = [
    # S, Hq, Hkv, d, dtype, b, k, shuffle
    (2048, 32, 8, 128, "bf16", 64, 1024, False),    # block kernel, 16 tiles
    (2304, 32, 8, 128, "bf16", 128, 2048, False),   # block kernel, b = 128, 32 tiles
    (2100, 16, 4, 128, "bf16", 16, 600, True),      # block kernel, ragged, shuffled
    (2000, 16, 4, 64, "bf16", 64, 777, False),      # block kernel, d = 64, ragged tile
    (2048, 16, 4, 128, "bf16", 1, 512, False),      # per-query kernel, 16 tiles
    (1500, 8, 2, 64, "bf16", 4, 700, True),         # per-query kernel, b = 4, shuffled
    (1200, 4, 2, 64, "f32", 1, 500, False),         # row-wise, fp32
    (700, 34, 2, 64, "bf16", 1, 300, False),        # row-wise, G = 17
    (600, 8, 2, 256, "bf16", 4, 400, False),        # per-query kernel, d = 256, b = 4
    (1500, 8, 2, 256, "bf16", 1, 700, True),        # per-query kernel, d = 256, shuffled
    (700, 34, 2, 256, "bf16", 1, 300, False),       # row-wise, d = 256, G = 17
    (600, 8, 2, 256, "bf16", 16, 400, False),       # block kernel, d = 256, 7 tiles
    (2048, 8, 2, 256, "bf16", 64, 1024, False),     # block kernel, d = 256, 16 tiles
    (2200, 8, 4, 256, "bf16", 16, 700, True),       # block kernel, d = 256, G = 2, shuffled
    (4200, 4, 2, 256, "bf16", 64, 3000, False),     # block kernel, d = 256, 47 tiles
    (4700, 4, 2, 64, "bf16", 64, 4500, True),       # b = 64 with k > 4096: per-query kernel
]


@pytest.mark.parametrize("case", SHARP_CASES, ids=lambda c: "-".join(map(str, c)))
def test_sparse_attention_sharp_multitile(case):
    S, Hq, Hkv, d, dtype, b, k, shuffle = case
    say(f"sparse sharp {case}")
    inp = make_inputs(S, Hq, Hkv, d, dtype=dtype, seed=S + k + 1, peaked=True, unit_v=True,
                      k_ramp=8.0)
    idx = make_support(S, b, k, seed=b + 1, shuffle=shuffle)
    p = B.Problem(S, Hq, Hkv, d, topk=k, block_q=b, dtype=dtype)
    o = torch.empty(S, Hq, d, dtype=inp.q.dtype, device="cuda")
    B.sp_sparse_gqa_attn(p, cuda(inp.q), cuda(inp.k), cuda(inp.v), cuda(idx), o)
    torch.cuda.synchronize()
    R = p.num_blocks
    blocks = sorted(set([0, 1, R // 2, R - 2, R - 1] +
                        np.random.default_rng(S).choice(R, 3).tolist()))
    rows = np.concatenate([np.arange(r * b, min(r * b + b, S)) for r in blocks if r >= 0])
    rows = rows[:: max(1, len(rows) // 384)]
    rise = logit_rise(inp, idx, b, rows[-8:], 64 if b >= 16 else 32)
    say(f"  later-tile logit maximum rises by {rise:.1f} (base 2) over the first tile")
    assert rise > 8
    check_attention(f64(o)[rows], *ref_sparse(inp, idx, b, rows=rows), dtype)


@pytest.mark.parametrize("dtype,b,d", [("f32", 16, 128), ("bf16", 64, 128), ("bf16", 16, 64),
                                       ("bf16", 128, 128), ("bf16", 1, 128), ("bf16", 4, 64)])
def test_sparse_attention_order_and_sentinels(dtype, b, d):
    """Permuting a support row and padding it with sentinels and positions
    past the sequence changes which entries share a tile, so the fp32 row
    maxima, the bf16-rounded weights and the summation order all differ
    between the two calls: each result is held to the derived bound against
    the oracle, and the two to twice that bound against each other."""
    S, Hq, Hkv, k = 300, 8, 2, 64
    say(f"sparse shuffled support {dtype} b={b} d={d}")
    inp = _inp(S, Hq, Hkv, d, dtype=dtype, seed=5, peaked=True)
    idx = make_support(S, b, k, seed=1)
    rng = np.random.default_rng(0)
    shuf = torch.from_numpy(np.stack([rng.permutation(r) for r in idx.numpy()]))
    pad = torch.cat([shuf, torch.full((shuf.shape[0], 9), -1, dtype=torch.int32),
                     torch.full((shuf.shape[0], 3), S + 50, dtype=torch.int32)], dim=1)
    outs = []
    for table in (idx, pad):
        p = B.Problem(S, Hq, Hkv, d, topk=table.shape[1], block_q=b, dtype=dtype)
        o = torch.empty(S, Hq, d, dtype=inp.q.dtype, device="cuda")
        B.sp_sparse_gqa_attn(p, cuda(inp.q), cuda(inp.k), cuda(inp.v), cuda(table.contiguous()),
                             o)
        outs.append(f64(o))
    ref, ref_abs = ref_sparse(inp, idx, b)
    check_attention(outs[1], ref, ref_abs, dtype, "shuffled vs oracle: ")
    check_attention(outs[1], outs[0], ref_abs, dtype, "shuffled vs sorted: ", factor=2.0)


# ----------------------------------------------------------------------- dense
DENSE_CASES = [
    # S, Hq, Hkv, d, dtype, sharp
    (1, 4, 2, 64, "f32", False),
    (77, 4, 2, 64, "f32", False),
    (300, 6, 3, 128, "f32", False),
    (300, 8, 2, 128, "bf16", False),
    (515, 32, 8, 128, "bf16", False),
    (260, 4, 4, 64, "bf16", False),
    (333, 8, 8, 128, "bf16", False),
    (333, 8, 1, 64, "bf16", False),
    (1100, 32, 8, 128, "bf16", False),
    (1100, 32, 8, 128, "bf16", True),      # rescale after the first key tile
    (900, 8, 2, 64, "bf16", True),
    (700, 4, 2, 64, "f32", True),
    (333, 8, 1, 256, "bf16", False),       # d = 256: one group of four waves
    (700, 16, 4, 256, "bf16", False),
    (1100, 8, 2, 256, "bf16", True),
]


@pytest.mark.parametrize("case", DENSE_CASES, ids=lambda c: "-".join(map(str, c)))
def test_dense_attention(case):
    S, Hq, Hkv, d, dtype, sharp = case
    say(f"dense {case}")
    if sharp:
        inp = make_inputs(S, Hq, Hkv, d, dtype=dtype, seed=S + 3, peaked=True, unit_v=True,
                          k_ramp=8.0)
    else:
        inp = _inp(S, Hq, Hkv, d, dtype=dtype, seed=S, peaked=(dtype == "f32"),
                   needles=min(S, 4))
    p = B.Problem(S, Hq, Hkv, d, dtype=dtype)
    o = torch.empty(S, Hq, d, dtype=inp.q.dtype, device="cuda")
    lse = torch.empty(S, Hq, device="cuda")
    lse2 = torch.empty(S, Hq, device="cuda")
    q, k, v = cuda(inp.q), cuda(inp.k), cuda(inp.v)
    B.sp_dense_attn(p, q, k, v, o, lse)
    B.sp_dense_attn(p, q, k, v, None, lse2)
    torch.cuda.synchronize()
    ref_o, ref_lse = oracle.dense(inp.q, inp.k, inp.v)
    ref_abs, _ = oracle.dense(inp.q, inp.k, inp.v.abs())
    check_attention(f64(o), ref_o, ref_abs, dtype)
    el = max_err(f64(lse), ref_lse)
    say(f"  lse err {el:.3e}")
    # lse carries the logits' own rounding, which grows with their size
    assert el <= (1e-5 if dtype == "f32" else 1e-4) * max(1.0, np.abs(ref_lse).max())
    # the normaliser-only call runs a separate instance of the same kernel
    # (no P.V product); its fp32 normalisers agree to a few ulps
    rel = ((lse - lse2).abs() / lse.abs().clamp_min(1.0)).max().item()
    say(f"  normaliser-only lse vs full: max rel diff {rel:.2e}")
    assert rel <= 2.0 ** -20


# ----------------------------------------------------------------------- top-k
TOPK_CASES = [
    # R-defining (S, b), k, W, kind
    (300, 1, 37, 0, "gauss"),
    (300, 1, 37, 5, "relu"),
    (300, 7, 64, 0, "coarse"),
    (300, 64, 100, 16, "gauss"),
    (300, 64, 100, 100, "gauss"),
    (300, 3, 1, 0, "coarse"),
    (300, 3, 1, 1, "relu"),
    (300, 1, 299, 0, "const"),
    (5000, 64, 512, 0, "relu"),
    (9000, 128, 2048, 128, "gauss"),
    (9000, 128, 700, 0, "coarse"),
    (20000, 64, 2048, 0, "const"),     # every key on the threshold: no compaction
    (30000, 64, 9000, 0, "gauss"),     # more chosen than the LDS staging holds
    (32768, 64, 2048, 0, "relu"),      # the 32K block shape, ReLU zeros
    (30000, 64, 512, 16, "coarse"),    # long rows of 16 levels: crowded bins
    (3000, 12, 300, 8, "relu"),        # 16-byte row loads, candidate counts 4 mod 16
    (4000, 4, 256, 4, "coarse"),       # 16-byte row loads, 4-query blocks
    (4999, 1, 64, 3, "relu"),          # rows not 16-byte aligned: tested loads
    (3001, 64, 500, 0, "gauss"),       # rows not 16-byte aligned, 64-query blocks
    (70000, 70000, 40000, 0, "const"), # streamed row: one thread's bins hold > 65535 keys
    (70000, 35000, 3000, 17, "relu"),  # streamed rows with ReLU zeros and a window
    (69996, 34998, 2048, 1, "coarse"), # streamed 16-byte loads, candidate counts 1 and 3 mod 4
    (70001, 35001, 3000, 5, "gauss"),  # streamed rows not 16-byte aligned: one key per load
]


@pytest.mark.parametrize("case", TOPK_CASES, ids=lambda c: "-".join(map(str, c)))
def test_topk(case):
    S, b, k, W, kind = case
    say(f"topk {case}")
    R = (S + b - 1) // b
    scores = make_scores(R, S, seed=S + k, kind=kind)
    p = B.Problem(S, 1, 1, 64, topk=k, block_q=b, local_window=W, dtype="f32")
    idx = torch.empty(R, k, dtype=torch.int32, device="cuda")
    B.sp_topk_select(p, cuda(scores), idx)
    torch.cuda.synchronize()
    lens = np.array([min(r * b + b, S) for r in range(R)])
    ref = oracle.topk(scores.numpy().astype(np.float64), lens, k, W)
    got = idx.cpu().numpy()
    check_rows_ascending(got, lens, k)
    assert np.array_equal(got, ref)   # same fp32 values: selection must be bit-exact


def test_topk_streamed_crowded_bins():
    """A streamed row (70000 candidates) whose top bins hold 66000 equal keys
    and whose k-th largest lies below them: the block scan of per-thread bin
    counts must carry counts above 65535 to the threads owning lower bins."""
    S, k = 70000, 68000
    say("topk streamed crowded bins")
    rng = np.random.default_rng(11)
    row = np.ones(S, dtype=np.float32)
    low = rng.choice(S, 4000, replace=False)
    row[low] = -1.0 - rng.random(4000).astype(np.float32)
    scores = torch.from_numpy(row[None, :].copy())
    p = B.Problem(S, 1, 1, 64, topk=k, block_q=S, dtype="f32")
    idx = torch.empty(1, k, dtype=torch.int32, device="cuda")
    B.sp_topk_select(p, cuda(scores), idx)
    torch.cuda.synchronize()
    ref = oracle.topk(scores.numpy().astype(np.float64), np.array([S]), k, 0)
    assert np.array_equal(idx.cpu().numpy(), ref)


@pytest.mark.parametrize("n_close", [200, 256, 257, 300])
def test_topk_keys_sharing_the_high_bits(n_close):
    """Rows whose k-th largest key shares its top 22 bits with n_close keys
    (values 1 + m 2^-23, m < 64: many exact ties): up to 256 such keys the
    threshold is searched among them directly, beyond that by a third radix
    pass. Both must match the oracle bit for bit."""
    S, k = 4096, 150
    say(f"topk keys sharing the high bits {n_close}")
    rng = np.random.default_rng(100 + n_close)
    rows = []
    for _ in range(3):
        row = rng.uniform(-1.0, 0.5, S).astype(np.float32)
        pos = rng.choice(S, n_close, replace=False)
        m = rng.integers(0, 64, n_close)
        row[pos] = (np.float32(1.0) + m.astype(np.float32) * np.float32(2.0 ** -23))
        rows.append(row)
    scores = torch.from_numpy(np.stack(rows))
    p = B.Problem(S, 1, 1, 64, topk=k, block_q=S, dtype="f32")
    # three rows of one block each: lay them out as a batch of three problems
    for r in range(3):
        idx = torch.empty(1, k, dtype=torch.int32, device="cuda")
        B.sp_topk_select(p, cuda(scores[r:r + 1].contiguous()), idx)
        torch.cuda.synchronize()
        ref = oracle.topk(scores[r:r + 1].numpy().astype(np.float64), np.array([S]), k, 0)
        assert np.array_equal(idx.cpu().numpy(), ref)


# --------------------------------------------------------------- indexer scores
INDEXER_CASES = [
    # S, d_idx, b, agg, relu, dtype
    (300, 64, 1, "max", 1, "bf16"),
    (301, 128, 1, "max", 1, "bf16"),
    (1100, 128, 1, "max", 0, "bf16"),
    (300, 128, 16, "max", 1, "bf16"),
    (300, 128, 64, "sum", 1, "bf16"),
    (300, 256, 64, "max", 0, "bf16"),
    (300, 64, 7, "sum", 0, "f32"),
    (1000, 128, 128, "max", 1, "bf16"),
    (333, 256, 1, "max", 1, "bf16"),    # per query, 32-key tiles: 8 rows per store, rows unaligned
    (2050, 64, 1, "max", 0, "bf16"),    # per query, three key chunks, ragged last tile
]


@pytest.mark.parametrize("case", INDEXER_CASES, ids=lambda c: "-".join(map(str, c)))
def test_indexer_scores(case):
    S, di, b, agg, relu, dtype = case
    say(f"indexer {case}")
    inp = _inp(S, 1, 1, 64, di=di, dtype=dtype, seed=di + b, needles=8)
    p = B.Problem(S, 1, 1, 64, index_dim=di, topk=8, block_q=b, agg=agg, relu=relu, dtype=dtype)
    R = p.num_blocks
    sc = torch.full((R, S), float("nan"), device="cuda")
    B.sp_indexer_scores(p, cuda(inp.q_idx), cuda(inp.k_idx), sc)
    torch.cuda.synchronize()
    ref = oracle.support_scores("indexer", range(R), b, q_idx=inp.q_idx, k_idx=inp.k_idx,
                                agg=agg, relu=bool(relu))
    got = sc.cpu().numpy().astype(np.float64)
    scale = np.abs(ref).max()
    for r in range(R):
        L = min(r * b + b, S)
        e = max_err(got[r, :L], ref[r, :L])
        assert e <= 2e-6 * scale * (b if agg == "sum" else 1), (r, e, scale)
        assert np.all(np.isnan(got[r, L:]))   # invalid tail untouched


# ------------------------------------------------------------------ oracle mass
MASS_CASES = [
    # S, Hq, Hkv, d, b, agg, dtype
    (200, 4, 2, 64, 1, "max", "f32"),
    (200, 4, 2, 64, 8, "max", "f32"),
    (300, 8, 2, 128, 64, "max", "bf16"),
    (300, 8, 2, 128, 16, "sum", "bf16"),
    (260, 32, 8, 128, 1, "max", "bf16"),
    (300, 16, 4, 64, 32, "sum", "bf16"),
    (1000, 32, 8, 128, 128, "max", "bf16"),
    (200, 8, 1, 64, 1, "max", "bf16"),
    (300, 8, 2, 256, 1, "max", "bf16"),    # d = 256: the 16-query kernel
    (700, 32, 8, 256, 64, "max", "bf16"),
    (500, 16, 4, 256, 16, "sum", "bf16"),
    (300, 12, 4, 256, 32, "max", "bf16"),  # Hq not a multiple of 8: row-wise
]


@pytest.mark.parametrize("case", MASS_CASES, ids=lambda c: "-".join(map(str, c)))
def test_oracle_mass(case):
    S, Hq, Hkv, d, b, agg, dtype = case
    say(f"mass {case}")
    inp = _inp(S, Hq, Hkv, d, dtype=dtype, seed=S + b, peaked=True, needles=4)
    p = B.Problem(S, Hq, Hkv, d, topk=8, block_q=b, agg=agg, dtype=dtype)
    q, k, v = cuda(inp.q), cuda(inp.k), cuda(inp.v)
    lse = torch.empty(S, Hq, device="cuda")
    B.sp_dense_attn(p, q, k, v, None, lse)
    R = p.num_blocks
    mass = torch.full((R, S), float("nan"), device="cuda")
    B.sp_oracle_support(p, q, k, lse, mass)
    torch.cuda.synchronize()
    ref = oracle.support_scores("oracle", range(R), b, q=inp.q, k=inp.k, agg=agg)
    got = mass.cpu().numpy().astype(np.float64)
    for r in range(R):
        L = min(r * b + b, S)
        e = max_err(got[r, :L], ref[r, :L])
        scale = np.abs(ref[r, :L]).max()
        assert e <= 1e-4 * scale, (r, e, scale)
        assert np.all(np.isnan(got[r, L:]))

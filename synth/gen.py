"""Seeded synthetic inputs: Q/K/V, head-collapsed indexer vectors, planted needles.

Recipe (one numpy PCG64 stream per call, fixed draw order):

1. Q [S,Hq,d], K [S,Hkv,d], V [S,Hkv,d] ~ N(0,1)/sqrt(d) (``peaked=True``
   drops the 1/sqrt(d), giving logits of unit spread instead of ~1/d).
2. q_idx, k_idx [S,d_idx] ~ N(0,1) (the indexer's post-normalisation,
   post-RoPE vectors of Section 6.3; the projection itself is not modelled).
3. Needles: n positions p_i (uniform without replacement, or stratified
   p_i = floor((i+u_i)*S/n)), each with a probe query r_i ~ U[p_i, S) and a
   probe head h_i ~ U[0, Hq). K[p_i, every KV head] = 3 * Q[r_i,h_i]/|Q[r_i,h_i]|.
   When an indexer is present and not ``untrained``, also
   k_idx[p_i] = 3*sqrt(d_idx) * q_idx[r_i]/|q_idx[r_i]|.
4. Everything is drawn in fp32 and rounded once to the storage dtype
   (bf16 by round-to-nearest-even through torch).

Two test-only shapes of the same draws: ``unit_v=True`` drops the 1/sqrt(d)
of V (outputs of order 1/sqrt(|support|) instead of 1/sqrt(d |support|)),
and ``k_ramp=g`` multiplies key row s by 1 + g*s/(S-1) before the needles
are planted, so later keys carry ever larger logits and an online softmax
must raise its running maximum long after its first tile.

Needle retrieval mirrors the needle-in-a-haystack task family the paper
evaluates on (Section 5.1); no benchmark item is reproduced.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np
import torch

_TORCH_DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclasses.dataclass
class Inputs:
    q: torch.Tensor
    k: torch.Tensor
    v: torch.Tensor
    q_idx: Optional[torch.Tensor]
    k_idx: Optional[torch.Tensor]
    needle_pos: np.ndarray    # [n] int64
    probe_query: np.ndarray   # [n] int64
    probe_head: np.ndarray    # [n] int64

    def to(self, device) -> "Inputs":
        mv = lambda t: None if t is None else t.to(device)
        return dataclasses.replace(self, q=mv(self.q), k=mv(self.k), v=mv(self.v),
                                   q_idx=mv(self.q_idx), k_idx=mv(self.k_idx))


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def make_inputs(seq_len: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                index_dim: int = 0, dtype: str = "bf16", needles: int = 0,
                stratified: bool = False, seed: int = 0, peaked: bool = False,
                untrained: bool = False, unit_v: bool = False, k_ramp: float = 0.0) -> Inputs:
    S, Hq, Hkv, d, di = seq_len, num_q_heads, num_kv_heads, head_dim, index_dim
    rng = _rng(seed)
    sd = 1.0 if peaked else 1.0 / np.sqrt(d)
    q = rng.standard_normal((S, Hq, d), dtype=np.float32) * np.float32(sd)
    k = rng.standard_normal((S, Hkv, d), dtype=np.float32) * np.float32(sd)
    v = rng.standard_normal((S, Hkv, d), dtype=np.float32)
    if not unit_v:
        v *= np.float32(1.0 / np.sqrt(d))
    if k_ramp:
        gain = 1.0 + k_ramp * np.arange(S, dtype=np.float64) / max(S - 1, 1)
        k *= gain.astype(np.float32)[:, None, None]
    qi = ki = None
    if di > 0:
        qi = rng.standard_normal((S, di), dtype=np.float32)
        ki = rng.standard_normal((S, di), dtype=np.float32)
    n = min(needles, S)
    if n > 0:
        if stratified:
            u = rng.random(n)
            pos = np.floor((np.arange(n) + u) * S / n).astype(np.int64)
            pos = np.minimum(pos, S - 1)
        else:
            pos = np.sort(rng.choice(S, size=n, replace=False)).astype(np.int64)
        probe_q = (pos + np.floor(rng.random(n) * (S - pos))).astype(np.int64)
        probe_q = np.minimum(probe_q, S - 1)
        probe_h = rng.integers(0, Hq, size=n).astype(np.int64)
        for p, r, h in zip(pos, probe_q, probe_h):
            u = q[r, h] / np.linalg.norm(q[r, h])
            k[p, :, :] = 3.0 * u[None, :]
            if di > 0 and not untrained:
                qn = qi[r] / np.linalg.norm(qi[r])
                ki[p] = 3.0 * np.sqrt(di) * qn
    else:
        pos = probe_q = probe_h = np.zeros(0, dtype=np.int64)
    td = _TORCH_DTYPES[dtype]
    cv = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(td)
    return Inputs(q=cv(q), k=cv(k), v=cv(v), q_idx=cv(qi), k_idx=cv(ki),
                  needle_pos=pos, probe_query=probe_q, probe_head=probe_h)


def make_scores(rows: int, seq_len: int, seed: int = 0, kind: str = "gauss") -> torch.Tensor:
    """Score rows [rows, seq_len] fp32 for exercising top-k on its own.

    kind: "gauss" (distinct values), "relu" (about half exact zeros, with some
    negative zeros), "coarse" (values on a grid of 16 levels, so many exact
    ties), "const" (every entry equal).
    """
    rng = _rng(seed)
    x = rng.standard_normal((rows, seq_len), dtype=np.float32)
    if kind == "relu":
        x = np.maximum(x, np.float32(0.0))
        neg0 = rng.random((rows, seq_len)) < 0.1
        x[neg0 & (x == 0)] = np.float32(-0.0)
    elif kind == "coarse":
        x = np.round(x * 4.0).astype(np.float32) / np.float32(4.0)
    elif kind == "const":
        x[:] = np.float32(0.5)
    elif kind != "gauss":
        raise ValueError(kind)
    return torch.from_numpy(np.ascontiguousarray(x))


def make_support(seq_len: int, block_q: int, topk: int, seed: int = 0,
                 shuffle: bool = False, random_rows=None) -> torch.Tensor:
    """A random support table [R, topk] int32 for exercising sparse attention alone.

    Row r draws min(topk, t1_r+1) distinct positions from [0, t1_r], where t1_r
    is the last query of selection block r, stores them ascending (or shuffled)
    and pads with -1. With ``random_rows`` (a list of row numbers) only those
    rows are drawn; every other row holds its m most recent positions, which
    keeps full-size tables cheap to make where only some rows are checked.
    """
    rng = _rng(seed)
    R = (seq_len + block_q - 1) // block_q
    out = np.full((R, topk), -1, dtype=np.int32)
    drawn = range(R) if random_rows is None else sorted(set(int(r) for r in random_rows))
    if random_rows is not None:
        t1s = np.minimum(np.arange(R) * block_q + block_q, seq_len) - 1
        for r in range(R):
            m = min(topk, int(t1s[r]) + 1)
            out[r, :m] = np.arange(t1s[r] - m + 1, t1s[r] + 1, dtype=np.int32)
    for r in drawn:
        t1 = min(r * block_q + block_q, seq_len) - 1
        m = min(topk, t1 + 1)
        sel = np.sort(rng.choice(t1 + 1, size=m, replace=False))
        if shuffle:
            sel = rng.permutation(sel)
        out[r, :m] = sel
    return torch.from_numpy(out)


def make_kl_rows(n: int, seq_len: int, seed: int = 0, rows=None, zero_frac: float = 0.0,
                 tail: float = float("nan"), device="cpu"):
    """Teacher rows P, student rows z [n, seq_len] fp32 and their query positions.

    Row i belongs to query t_i (``rows``, or uniform in [0, seq_len)). On
    s <= t_i, P is u^3 for u ~ U(0,1) with a fraction ``zero_frac`` set to
    exact zeros, normalised to sum 1 (a row drawn all zero puts its mass on
    position 0); z ~ N(0, 4). Entries after t_i hold ``tail`` (NaN by
    default) so any read of them shows. Drawn with a seeded torch generator
    on ``device``, so full-size rows can be made where they are used.
    """
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    if rows is None:
        rows = torch.randint(0, seq_len, (n,), generator=g, device=device)
    rows = torch.as_tensor(rows, device=device).to(torch.int64)
    s = torch.arange(seq_len, device=device)
    valid = s[None, :] <= rows[:, None]
    u = torch.rand(n, seq_len, generator=g, device=device) ** 3
    if zero_frac > 0:
        drop = torch.rand(n, seq_len, generator=g, device=device) < zero_frac
        u = torch.where(drop, torch.zeros((), device=device), u)
    u = torch.where(valid, u, torch.zeros((), device=device))
    empty = u.sum(1) == 0
    u[:, 0] = torch.where(empty, torch.ones((), device=device), u[:, 0])
    P = u / u.sum(1, keepdim=True)
    z = torch.randn(n, seq_len, generator=g, device=device) * 2.0
    fill = torch.full((), tail, device=device)
    P = torch.where(valid, P, fill).to(torch.float32).contiguous()
    z = torch.where(valid, z, fill).to(torch.float32).contiguous()
    return rows.to(torch.int32), P, z


def make_projection_inputs(seq_len: int, d_model: int, index_dim: int, seed: int = 0):
    """Hidden states and random indexer-projection weights (the trained ones
    are not released): x [S, d_model] ~ N(0,1), W_Q and W_K [d_idx, d_model]
    ~ N(0, 1/d_model), all rounded to bf16; LayerNorm gamma ~ 1 + N(0, 0.01)
    and beta ~ N(0, 0.01) in fp32. Returns (x, w_q, w_k, gamma, beta)."""
    rng = _rng(seed)
    x = rng.standard_normal((seq_len, d_model), dtype=np.float32)
    sd = np.float32(1.0 / np.sqrt(d_model))
    wq = rng.standard_normal((index_dim, d_model), dtype=np.float32) * sd
    wk = rng.standard_normal((index_dim, d_model), dtype=np.float32) * sd
    gamma = (1.0 + 0.1 * rng.standard_normal(index_dim)).astype(np.float32)
    beta = (0.1 * rng.standard_normal(index_dim)).astype(np.float32)
    bf = lambda a: torch.from_numpy(a).to(torch.bfloat16)
    return bf(x), bf(wq), bf(wk), torch.from_numpy(gamma), torch.from_numpy(beta)


def make_index_vectors(seq_len: int, index_dim: int, seed: int = 0, kind: str = "gauss"):
    """Indexer vectors q_idx, k_idx [S, d_idx] in bf16 for exercising the
    scorer and selection on their own. kind "gauss": N(0,1); "ternary":
    entries in {-1, 0, 1}, so scores are integers and exact ties are common."""
    rng = _rng(seed)
    if kind == "gauss":
        q = rng.standard_normal((seq_len, index_dim), dtype=np.float32)
        k = rng.standard_normal((seq_len, index_dim), dtype=np.float32)
    elif kind == "ternary":
        q = rng.integers(-1, 2, size=(seq_len, index_dim)).astype(np.float32)
        k = rng.integers(-1, 2, size=(seq_len, index_dim)).astype(np.float32)
    else:
        raise ValueError(kind)
    bf = lambda a: torch.from_numpy(a).to(torch.bfloat16)
    return bf(q), bf(k)

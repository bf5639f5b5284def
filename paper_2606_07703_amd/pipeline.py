"""The three call sequences of the library, with outputs allocated by torch.

* ``indexer_prefill`` — Algorithm 2, scoring, selection and sparse prefill: indexer scores, top-k,
  sparse GQA attention.
* ``oracle_prefill`` — Algorithm 1, dense pass, selection and restricted recomputation: dense normalisers, head-averaged
  mass, top-k, sparse GQA attention.
* ``dense_prefill`` — Section 3 dense causal GQA attention.

``Buffers`` pre-allocates every output once so that repeated calls (the
benchmark's timed steps) allocate nothing.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

from .binding import (TORCH_DTYPE, Problem, sp_dense_attn, sp_indexer_scores,
                      sp_oracle_support, sp_sparse_gqa_attn, sp_topk_select)


@dataclasses.dataclass
class Buffers:
    o: torch.Tensor
    scores: torch.Tensor
    idx: torch.Tensor
    lse: Optional[torch.Tensor] = None

    @staticmethod
    def for_problem(p: Problem, device="cuda", oracle: bool = False) -> "Buffers":
        dt = TORCH_DTYPE[p.dtype]
        o = torch.empty(p.seq_len, p.num_q_heads, p.head_dim, dtype=dt, device=device)
        scores = torch.empty(p.table_rows + (p.seq_len,), dtype=torch.float32, device=device)
        idx = torch.empty(p.table_rows + (p.topk,), dtype=torch.int32, device=device)
        lse = (torch.empty(p.seq_len, p.num_q_heads, dtype=torch.float32, device=device)
               if oracle else None)
        return Buffers(o=o, scores=scores, idx=idx, lse=lse)


def indexer_prefill(p: Problem, q, k, v, q_idx, k_idx, buf: Optional[Buffers] = None,
                    stream=None) -> Buffers:
    buf = buf or Buffers.for_problem(p, q.device)
    sp_indexer_scores(p, q_idx, k_idx, buf.scores, stream)
    sp_topk_select(p, buf.scores, buf.idx, None, stream)
    sp_sparse_gqa_attn(p, q, k, v, buf.idx, buf.o, stream)
    return buf


def oracle_prefill(p: Problem, q, k, v, buf: Optional[Buffers] = None, stream=None) -> Buffers:
    buf = buf or Buffers.for_problem(p, q.device, oracle=True)
    sp_dense_attn(p, q, k, v, None, buf.lse, stream)
    sp_oracle_support(p, q, k, buf.lse, buf.scores, stream)
    sp_topk_select(p, buf.scores, buf.idx, None, stream)
    sp_sparse_gqa_attn(p, q, k, v, buf.idx, buf.o, stream)
    return buf


def dense_prefill(p: Problem, q, k, v, o=None, lse=None, stream=None):
    if o is None:
        o = torch.empty(p.seq_len, p.num_q_heads, p.head_dim, dtype=TORCH_DTYPE[p.dtype],
                        device=q.device)
    sp_dense_attn(p, q, k, v, o, lse, stream)
    return o

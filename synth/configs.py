"""Workload shapes for the sparse GQA prefill path.

Each workload is a synthetic, Qwen-like GQA layer: sequence length S, query
heads Hq, KV heads Hkv, head dim d, indexer dim d_idx, top-k budget k,
selection-block size b_sel, forced local window W, block aggregation rule and
storage dtype. Budgets and lengths follow the paper's evaluated ranges
(Section 5.1: 4K..100K contexts, top-k 256..2048; Section 8, Finding 3: top-k up to 1024
at 32K; b_sel in {1, 64} in Section 5.1). "100K" is 102,400 tokens: only that
length reproduces the 96.0% causal sparsity printed in Table 2.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    seq_len: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    index_dim: int          # 0 = no indexer (oracle mode only)
    topk: int
    block_q: Tuple[int, ...]  # selection-block sizes run on this workload
    local_window: int
    agg: Tuple[str, ...]    # "max" (paper) and/or "sum"
    dtype: str              # "f32" | "bf16"
    needles: int
    stratified: bool = False
    modes: Tuple[str, ...] = ("indexer",)
    seed: int = 0
    description: str = ""

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


WORKLOADS = {
    "oracle_tiny_512": Workload(
        name="oracle_tiny_512", seq_len=512, num_q_heads=4, num_kv_heads=2,
        head_dim=64, index_dim=0, topk=64, block_q=(1,), local_window=0,
        agg=("max",), dtype="f32", needles=8, modes=("oracle",), seed=1,
        description="oracle mode, S=512, 4/2 heads, d=64, fp32, per-query top-64"),
    "indexer_4k": Workload(
        name="indexer_4k", seq_len=4096, num_q_heads=16, num_kv_heads=4,
        head_dim=128, index_dim=64, topk=512, block_q=(1,), local_window=0,
        agg=("max",), dtype="bf16", needles=32, modes=("indexer", "dense"), seed=2,
        description="indexer path, S=4096, 16/4 heads, d=128, d_idx=64, per-query top-512"),
    "block_16k": Workload(
        name="block_16k", seq_len=16384, num_q_heads=32, num_kv_heads=8,
        head_dim=128, index_dim=128, topk=2048, block_q=(64,), local_window=128,
        agg=("sum", "max"), dtype="bf16", needles=64, modes=("indexer", "dense"), seed=3,
        description="block-shared selection, S=16384, 32/8 heads, d=128, d_idx=128, "
                    "top-2048 per 64-query block, 128-token local window"),
    "headline_32k": Workload(
        name="headline_32k", seq_len=32768, num_q_heads=32, num_kv_heads=8,
        head_dim=128, index_dim=128, topk=2048, block_q=(64, 1), local_window=0,
        agg=("max",), dtype="bf16", needles=128, modes=("indexer", "dense", "oracle"), seed=4,
        description="S=32768, 32/8 heads, d=128, d_idx=128, top-2048, "
                    "per-query and 64-query-block selection, dense and oracle modes"),
    "stress_100k": Workload(
        name="stress_100k", seq_len=102400, num_q_heads=32, num_kv_heads=8,
        head_dim=128, index_dim=128, topk=4096, block_q=(128,), local_window=0,
        agg=("max",), dtype="bf16", needles=256, stratified=True,
        modes=("indexer", "dense"), seed=5,
        description="S=102400, 32/8 heads, d=128, d_idx=128, top-4096 per 128-query block, "
                    "256 stratified needles, plus an untrained-indexer variant"),
    # not one of the paper's measured configurations: the 32K shape at the
    # head dim of the paper's Qwen3.5 models (Section 6.3: d_idx = 256 equals
    # it), timing the head_dim-256 kernels
    "head256_32k": Workload(
        name="head256_32k", seq_len=32768, num_q_heads=32, num_kv_heads=8,
        head_dim=256, index_dim=256, topk=2048, block_q=(64,), local_window=0,
        agg=("max",), dtype="bf16", needles=128, modes=("indexer", "dense"), seed=6,
        description="S=32768, 32/8 heads, d=256, d_idx=256, top-2048 per 64-query block"),
}


def get_workload(name: str, seq_len: Optional[int] = None) -> Workload:
    w = WORKLOADS[name]
    if seq_len is not None:
        w = dataclasses.replace(w, seq_len=seq_len)
    return w

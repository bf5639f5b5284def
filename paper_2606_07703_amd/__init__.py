"""MI355X (gfx950) causal top-k sparse GQA prefill.

The compute lives in ``libsparse_prefill.so`` (hand-written HIP kernels behind
the C ABI declared in ``include/sparse_prefill.h``); this package is its thin
binding. Importing it does not load the library; the first call does, and
raises if the library has not been built.
"""
from .binding import (Problem, SparsePrefillError, load, sp_dense_attn,  # noqa: F401
                      sp_indexer_scores, sp_oracle_support, sp_sparse_gqa_attn,
                      sp_topk_select, sp_version, sp_workspace_bytes)
from .pipeline import Buffers, dense_prefill, indexer_prefill, oracle_prefill  # noqa: F401

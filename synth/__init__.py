"""Seeded synthetic inputs for causal top-k sparse GQA prefill.

This package is shared by the tests, the benchmark and the oracle's callers.
It holds only input generation (random draws, needle planting, rounding to
the storage dtype) and the workload shape registry; none of the method's
arithmetic lives here.
"""
from .configs import WORKLOADS, Workload, get_workload  # noqa: F401
from .gen import (make_index_vectors, make_inputs, make_kl_rows, make_projection_inputs,  # noqa: F401
                  make_scores, make_support, Inputs)

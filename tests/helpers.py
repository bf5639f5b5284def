"""Comparison rules shared by the GPU parity tests.

Selected sets: for a row with more than k causal positions, let v_k and
v_{k+1} be the oracle's k'-th and (k'+1)-th largest candidate values (fp64,
k' = k minus the forced window). If (v_k - v_{k+1})/|v_k| > 1e-4 the GPU's
set must equal the oracle's exactly; otherwise the GPU's set must be valid
within 1e-4 relative: everything clearly above v_k is chosen, nothing chosen
is clearly below it, and exactly k' candidates are chosen. Rows with at most
k positions must match exactly. Every GPU row must also be ascending,
distinct and padded with -1.
"""
import sys

import numpy as np
import torch

import oracle

GAP = 1e-4


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def cuda(t):
    return None if t is None else t.to("cuda")


def f64(t):
    return t.detach().to("cpu").to(torch.float64).numpy()


def check_rows_ascending(idx: np.ndarray, lens: np.ndarray, k: int) -> None:
    for row, L in zip(idx, lens):
        m = int((row >= 0).sum())
        assert m == min(L, k), (m, L, k)
        assert np.all(row[m:] == -1)
        assert np.all(np.diff(row[:m]) > 0)
        assert m == 0 or (row[0] >= 0 and row[m - 1] < L)


def compare_support(gpu_row: np.ndarray, orc_row: np.ndarray, Y: np.ndarray, L: int, k: int,
                    window: int = 0) -> str:
    """Returns 'exact' or 'tolerant' (which rule applied); asserts on failure."""
    if L <= k:
        assert np.array_equal(gpu_row, orc_row)
        return "exact"
    Wf = min(window, k)
    kp = k - Wf
    forced = set(range(L - Wf, L))
    g = set(int(s) for s in gpu_row if s >= 0)
    assert forced <= g
    info = oracle.topk_gap(Y, L, k, window)
    if info is None:
        assert np.array_equal(gpu_row, orc_row)
        return "exact"
    vk, vk1, gap = info
    if gap > GAP:
        assert np.array_equal(gpu_row, orc_row), (vk, vk1, gap)
        return "exact"
    cand = g - forced
    assert len(cand) == kp
    tol = GAP * max(abs(vk), 1e-30)
    y = Y[: L - Wf]
    must = set(np.nonzero(y > vk + tol)[0].tolist())
    assert must <= cand
    assert all(y[s] >= vk - tol for s in cand)
    return "tolerant"


def max_err(a: np.ndarray, b: np.ndarray) -> float:
    return float(np.abs(a - b).max()) if a.size else 0.0


def tol_for(dtype: str) -> float:
    return 1e-5 if dtype == "f32" else 2e-2

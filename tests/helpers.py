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
    """The stated absolute bound on attention outputs: bf16 2e-2, fp32 1e-5."""
    return 1e-5 if dtype == "f32" else 2e-2


def attn_bound(ref: np.ndarray, ref_abs: np.ndarray, dtype: str) -> np.ndarray:
    """Per-element bound on |o_gpu - o| derived from the kernels' arithmetic.

    o = sum_s w_s v_s with softmax weights w_s over the usable support; A =
    sum_s w_s |v_s| is the same attention taken over |V| (``ref_abs``).
    bf16: each unnormalised weight exp2(l_s - m) is computed in fp32 and
    rounded once to bf16 for the P.V product (relative error <= u = 2^-8,
    while the normaliser sums the unrounded fp32 values), products of bf16
    operands are exact in fp32 and summed in fp32, and o is rounded once to
    bf16 (<= u |o|). So |o_gpu - o| <= u A + u |o| + (fp32 terms of order
    2^-24 d); the check allows twice that. fp32: no bf16 rounding anywhere;
    the logits carry fp32 rounding of order d * 2^-24 * sum |q_c k_c| *
    scale, which the relative terms below cover with a wide margin.
    Unlike a flat absolute bound this scales with the outputs: an all-zero
    or support-mean output fails it wherever the attention is not uniform.
    """
    if dtype == "f32":
        return 1e-4 * ref_abs + 1e-5 * np.abs(ref) + 1e-7
    u = 2.0 ** -8
    return 2 * u * ref_abs + 2 * u * np.abs(ref) + 1e-6


def check_attention(got: np.ndarray, ref: np.ndarray, ref_abs: np.ndarray, dtype: str,
                    label: str = "", factor: float = 1.0) -> float:
    """Asserts the stated absolute bound and the derived per-element bound
    (``factor`` times it, e.g. 2 for two GPU results each within it); returns
    the worst err/bound ratio. The stated bound (bf16 2e-2, fp32 1e-5) is
    absolute for outputs up to 1 in magnitude (every workload's outputs stay
    below 0.05) and relative above that: the unit-spread V of the sharp test
    inputs gives outputs up to about 5, where one bf16 rounding of the output
    alone reaches 2^-8 * 4 = 0.0156."""
    err = np.abs(got - ref)
    bound = factor * attn_bound(ref, ref_abs, dtype)
    ratio = float((err / bound).max()) if err.size else 0.0
    rel_rms = float(np.sqrt((err ** 2).mean() / max((ref ** 2).mean(), 1e-300))) if err.size \
        else 0.0
    say(f"  {label}max abs err {err.max() if err.size else 0:.3e}, max|ref| "
        f"{np.abs(ref).max() if ref.size else 0:.3e}, rms err/rms ref {rel_rms:.2e}, "
        f"worst err/bound {ratio:.3f}")
    assert err.size == 0 or (err <= factor * tol_for(dtype) * np.maximum(1.0, np.abs(ref))).all()
    assert ratio <= 1.0, (ratio, label)
    return ratio


def logit_rise(inp, idx, b, rows, tile):
    """Largest rise, in base-2 units, of a later support tile's maximum scaled
    logit over the first tile's, among the given query rows and every head.
    Support tiles are the row's usable entries in table order, `tile` at a
    time (how the MFMA kernels walk them). Shows that a case reaches the
    online-softmax rescale after the first tile (a rise above 8)."""
    Hq, d = inp.q.shape[1], inp.q.shape[2]
    G = Hq // inp.k.shape[1]
    sl2 = 1.4426950408889634 / np.sqrt(d)
    table = idx.numpy()
    best = -np.inf
    for t in rows:
        row = table[t // b]
        use = row[(row >= 0) & (row <= t)]
        if len(use) <= tile:
            continue
        qt = inp.q[int(t)].double().numpy()
        kt = inp.k[torch.as_tensor(use, dtype=torch.long)].double().numpy()
        for h in range(Hq):
            lg = (kt[:, h // G] @ qt[h]) * sl2
            tiles = [lg[i:i + tile].max() for i in range(0, len(lg), tile)]
            best = max(best, max(tiles[1:]) - tiles[0])
    return best

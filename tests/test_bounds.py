"""The attention comparison bound separates right from plausibly wrong (CPU).

The GPU parity tests hold outputs to a per-element bound derived from the
kernels' arithmetic (``helpers.attn_bound``). Here, on the oracle alone:
outputs carrying exactly the modelled rounding (bf16 weights, bf16 output)
pass and an all-zero output fails, on the sharp multi-tile inputs and on
the near-uniform inputs of the named workloads' distribution. The support
mean of V (the result of a dropped q.k term) fails on the sharp inputs
only: with logits of spread about 1/d the softmax weights are within about
1% of uniform, so no bound can tell the two apart there, which is why every
kernel also runs the sharp variants.
"""
import numpy as np
import pytest
import torch

import oracle
from synth import make_inputs, make_support

from helpers import check_attention


def _bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(torch.float32).to(torch.bfloat16) \
        .to(torch.float64).numpy()


def _modelled(inp, idx, b, rows):
    """Restricted attention with the kernels' roundings applied in numpy:
    each unnormalised weight rounded to bf16 (normaliser from the unrounded
    ones), the output rounded to bf16."""
    q, k, v = (t.double().numpy() for t in (inp.q, inp.k, inp.v))
    Hq, d = q.shape[1], q.shape[2]
    G = Hq // k.shape[1]
    out = np.zeros((len(rows), Hq, d))
    for i, t in enumerate(rows):
        row = idx[t // b]
        use = row[(row >= 0) & (row <= t)]
        for h in range(Hq):
            lg = k[use, h // G] @ q[t, h] / np.sqrt(d)
            p = np.exp(lg - lg.max()).astype(np.float32)
            out[i, h] = (_bf16(p) @ v[use, h // G]) / p.astype(np.float64).sum()
    return _bf16(out)


@pytest.mark.parametrize("sharp", [True, False])
def test_bound_accepts_modelled_rounding_and_rejects_mistakes(sharp):
    S, Hq, Hkv, d, b, k = 640, 8, 2, 128, 64, 300
    inp = make_inputs(S, Hq, Hkv, d, dtype="bf16", seed=21, peaked=sharp, unit_v=sharp,
                      k_ramp=8.0 if sharp else 0.0)
    idx = make_support(S, b, k, seed=3).numpy()
    rows = np.arange(320, S, 7)
    ref = oracle.sparse(inp.q, inp.k, inp.v, idx, b, rows=rows)
    ref_abs = oracle.sparse(inp.q, inp.k, inp.v.abs(), idx, b, rows=rows)
    check_attention(_modelled(inp, idx, b, rows), ref, ref_abs, "bf16")
    with pytest.raises(AssertionError):
        check_attention(np.zeros_like(ref), ref, ref_abs, "bf16")
    mean_v = oracle.sparse(torch.zeros_like(inp.q), inp.k, inp.v, idx, b, rows=rows)
    if sharp:
        with pytest.raises(AssertionError):
            check_attention(mean_v, ref, ref_abs, "bf16")
    else:
        check_attention(mean_v, ref, ref_abs, "bf16")

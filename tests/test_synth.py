"""The seeded generator: determinism and planted structure."""
import numpy as np
import torch

from synth import make_inputs, make_scores, make_support


def test_same_seed_same_bytes():
    a = make_inputs(256, 4, 2, 64, index_dim=32, dtype="bf16", needles=8, seed=3)
    b = make_inputs(256, 4, 2, 64, index_dim=32, dtype="bf16", needles=8, seed=3)
    c = make_inputs(256, 4, 2, 64, index_dim=32, dtype="bf16", needles=8, seed=4)
    for x, y in [(a.q, b.q), (a.k, b.k), (a.v, b.v), (a.q_idx, b.q_idx), (a.k_idx, b.k_idx)]:
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))
    assert not torch.equal(a.q, c.q)
    assert np.array_equal(a.needle_pos, b.needle_pos)


def test_needles_planted():
    inp = make_inputs(512, 8, 2, 64, index_dim=64, dtype="f32", needles=16, seed=1)
    q, k, qi, ki = inp.q.numpy(), inp.k.numpy(), inp.q_idx.numpy(), inp.k_idx.numpy()
    assert len(set(inp.needle_pos.tolist())) == 16
    for p, r, h in zip(inp.needle_pos, inp.probe_query, inp.probe_head):
        assert r >= p
        u = q[r, h] / np.linalg.norm(q[r, h])
        for j in range(2):
            assert np.allclose(k[p, j], 3 * u, atol=1e-6)
        assert np.allclose(ki[p], 3 * np.sqrt(64) * qi[r] / np.linalg.norm(qi[r]), atol=1e-5)


def test_stratified_and_untrained():
    inp = make_inputs(1000, 2, 1, 16, index_dim=16, needles=10, stratified=True, seed=2,
                      untrained=True)
    assert np.array_equal(inp.needle_pos // 100, np.arange(10))
    # untrained: indexer keys are not planted
    raw = make_inputs(1000, 2, 1, 16, index_dim=16, needles=0, seed=2)
    assert inp.k_idx.shape == raw.k_idx.shape


def test_scores_and_supports():
    z = make_scores(4, 100, kind="relu").numpy()
    assert (z == 0).mean() > 0.3 and np.signbit(z[z == 0]).any()
    idx = make_support(100, 8, 16, seed=0).numpy()
    assert idx.shape == (13, 16)
    for r, row in enumerate(idx):
        t1 = min(r * 8 + 8, 100) - 1
        m = min(16, t1 + 1)
        assert np.all(np.diff(row[:m]) > 0) and row[:m].max() <= t1
        assert np.all(row[m:] == -1)

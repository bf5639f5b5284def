"""Pins for the oracle's KL objective, indexer front end and per-group supports (no GPU).

Each check ties the fp64 oracle to something other than itself: scipy's
relative entropy, closed forms, finite differences, torch's CPU LayerNorm,
numpy's matmul, and the algebraic properties of rotary position encoding.
"""
import numpy as np
import pytest
import scipy.special as ssp
import scipy.stats as sst
import torch

import oracle


def _rows_pz(n, S, seed, zero_frac=0.0):
    rng = np.random.default_rng(seed)
    rows = rng.integers(0, S, size=n).astype(np.int32)
    rows[0] = S - 1
    P = np.zeros((n, S))
    z = rng.normal(size=(n, S)) * 2.0
    for i, t in enumerate(rows):
        p = rng.dirichlet(np.ones(t + 1))
        if zero_frac > 0:
            p[rng.random(t + 1) < zero_frac] = 0.0
            if p.sum() == 0:
                p[0] = 1.0
            p /= p.sum()
        P[i, : t + 1] = p
        P[i, t + 1:] = rng.random(S - t - 1)        # beyond t: must be ignored
    return rows, P, z


# ----------------------------------------------------------------------- KL
@pytest.mark.parametrize("zero_frac", [0.0, 0.3])
def test_kl_matches_scipy_relative_entropy(zero_frac):
    rows, P, z = _rows_pz(9, 40, seed=1, zero_frac=zero_frac)
    kl, _ = oracle.kl(P, z, rows)
    for i, t in enumerate(rows):
        q = ssp.softmax(z[i, : t + 1])
        assert kl[i] == pytest.approx(sst.entropy(P[i, : t + 1], q), rel=1e-12, abs=1e-14)


def test_kl_zero_when_student_matches_teacher():
    rows, P, _ = _rows_pz(6, 30, seed=2)
    z = np.where(P > 0, np.log(np.maximum(P, 1e-300)), -5.0) + 3.7   # shift-invariant
    kl, grad = oracle.kl(P, z, rows)
    assert np.max(np.abs(kl)) < 1e-12
    assert np.max(np.abs(grad)) < 1e-12


def test_kl_one_hot_teacher_closed_form():
    S = 25
    rng = np.random.default_rng(3)
    rows = np.array([0, 7, 24], dtype=np.int32)
    z = rng.normal(size=(3, S))
    P = np.zeros((3, S))
    star = [0, 3, 20]
    for i, s in enumerate(star):
        P[i, s] = 1.0
    kl, _ = oracle.kl(P, z, rows)
    for i, t in enumerate(rows):
        assert kl[i] == pytest.approx(ssp.logsumexp(z[i, : t + 1]) - z[i, star[i]], rel=1e-12)


def test_kl_gradient_matches_finite_differences():
    rows, P, z = _rows_pz(3, 7, seed=4)
    _, grad = oracle.kl(P, z, rows)
    h = 1e-6
    for i in range(3):
        for s in range(7):
            zp, zm = z.copy(), z.copy()
            zp[i, s] += h
            zm[i, s] -= h
            fd = (oracle.kl(P, zp, rows)[0].mean() - oracle.kl(P, zm, rows)[0].mean()) / (2 * h)
            assert grad[i, s] == pytest.approx(fd, abs=1e-8)


def test_kl_ignores_entries_after_t_and_bad_rows():
    rows, P, z = _rows_pz(5, 20, seed=5)
    kl, grad = oracle.kl(P, z, rows)
    P2, z2 = P.copy(), z.copy()
    for i, t in enumerate(rows):
        P2[i, t + 1:] = 7.0
        z2[i, t + 1:] = -9.0
    kl2, grad2 = oracle.kl(P2, z2, rows)
    assert np.array_equal(kl, kl2) and np.array_equal(grad, grad2)
    for i, t in enumerate(rows):
        assert np.all(grad[i, t + 1:] == 0.0)
        # the gradient of each row sums to zero (softmax sums to one)
        assert abs(grad[i].sum()) < 1e-14
    bad = rows.copy()
    bad[1], bad[2] = -1, 20
    kl3, grad3 = oracle.kl(P, z, bad)
    assert kl3[1] == 0.0 and kl3[2] == 0.0
    assert np.all(grad3[1] == 0.0) and np.all(grad3[2] == 0.0)


def test_kl_nonnegative_for_distributions():
    rows, P, z = _rows_pz(30, 50, seed=6, zero_frac=0.2)
    kl, _ = oracle.kl(P, z, rows)
    assert np.all(kl >= -1e-14)


# ---------------------------------------------------------------- front end
def _proj_inputs(S, dm, di, seed, affine=True):
    rng = np.random.default_rng(seed)
    x = rng.normal(size=(S, dm))
    wq = rng.normal(size=(di, dm)) / np.sqrt(dm)
    wk = rng.normal(size=(di, dm)) / np.sqrt(dm)
    gamma = 1.0 + 0.1 * rng.normal(size=di) if affine else np.ones(di)
    beta = 0.1 * rng.normal(size=di) if affine else np.zeros(di)
    return x, wq, wk, gamma, beta


def test_project_position_zero_is_gemm_and_layernorm():
    x, wq, wk, gamma, beta = _proj_inputs(9, 48, 16, seed=7)
    q0, k0 = oracle.project(x, wq, wk, gamma, beta, rows=[0], pos0=0)
    assert np.allclose(q0[0], wq @ x[0], rtol=1e-12, atol=1e-12)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(wk @ x[0]), (16,),
                                         torch.from_numpy(gamma), torch.from_numpy(beta),
                                         eps=1e-6).numpy()
    assert np.allclose(k0[0], ref, rtol=1e-10, atol=1e-12)


def test_project_layernorm_standardises_keys():
    x, wq, wk, gamma, beta = _proj_inputs(5, 32, 16, seed=8, affine=False)
    # position 0 so RoPE is the identity
    _, k0 = oracle.project(x, wq, wk, gamma, beta, rows=[0], pos0=0)
    assert abs(k0[0].mean()) < 1e-12
    assert k0[0].var() == pytest.approx(1.0, rel=1e-4)   # var / (var + eps)


def test_rope_is_a_rotation_of_each_pair():
    # d_idx = 2: a single pair rotated by the angle pos * theta^0 = pos
    x, wq, wk, gamma, beta = _proj_inputs(6, 4, 2, seed=9)
    q, _ = oracle.project(x, wq, wk, gamma, beta, pos0=0)
    for t in range(6):
        a = wq @ x[t]
        c, s = np.cos(t), np.sin(t)
        assert np.allclose(q[t], [a[0] * c - a[1] * s, a[1] * c + a[0] * s], atol=1e-12)


def test_rope_preserves_norms_and_depends_on_relative_position():
    S, dm, di = 12, 40, 32
    x, wq, wk, gamma, beta = _proj_inputs(S, dm, di, seed=10)
    q, k = oracle.project(x, wq, wk, gamma, beta, pos0=0)
    q2, k2 = oracle.project(x, wq, wk, gamma, beta, pos0=1000)
    raw_q = x @ wq.T
    assert np.allclose(np.linalg.norm(q, axis=1), np.linalg.norm(raw_q, axis=1), rtol=1e-12)
    # scores depend on the position difference only: shifting every position
    # by 1000 leaves the score matrix unchanged, while the vectors move
    assert np.allclose(q @ k.T, q2 @ k2.T, rtol=1e-9, atol=1e-9)
    assert not np.allclose(q[1:], q2[1:])


def test_rope_frequency_schedule():
    # the pair c rotates by pos * theta^(-2c/d): with x such that W_Q x_t is the
    # unit vector e_c at every t, q_idx[t] traces that angle
    S, di = 5, 8
    for c in range(di // 2):
        x = np.ones((S, 1))
        wq = np.zeros((di, 1))
        wq[c, 0] = 1.0
        wk = np.ones((di, 1))
        q, _ = oracle.project(x, wq, wk, np.ones(di), np.zeros(di), pos0=3, theta=500.0)
        for t in range(S):
            ang = (3 + t) * 500.0 ** (-2.0 * c / di)
            assert q[t, c] == pytest.approx(np.cos(ang), abs=1e-12)
            assert q[t, c + di // 2] == pytest.approx(np.sin(ang), abs=1e-12)


# ------------------------------------------------------ per-KV-group supports
def _qkv(S, Hq, Hkv, d, seed):
    rng = np.random.default_rng(seed)
    return (rng.normal(size=(S, Hq, d)), rng.normal(size=(S, Hkv, d)),
            rng.normal(size=(S, Hkv, d)))


def test_group_mass_of_one_head_is_its_softmax_row():
    S, H, d = 30, 3, 8
    q, k, _ = _qkv(S, H, H, d, seed=11)          # G = 1: each group is one head
    rows = np.array([0, 5, 29])
    for j in range(H):
        P = oracle.mass(q, k, rows=rows, group=j)
        for i, t in enumerate(rows):
            ref = ssp.softmax(q[t, j] @ k[: t + 1, j].T / np.sqrt(d))
            assert np.allclose(P[i, : t + 1], ref, rtol=1e-12, atol=1e-15)


def test_group_masses_average_to_the_head_averaged_mass():
    S, Hq, Hkv, d = 40, 8, 4, 16
    q, k, _ = _qkv(S, Hq, Hkv, d, seed=12)
    rows = np.arange(0, S, 3)
    full = oracle.mass(q, k, rows=rows)
    groups = np.stack([oracle.mass(q, k, rows=rows, group=j) for j in range(Hkv)])
    assert np.allclose(groups.mean(axis=0), full, rtol=1e-12, atol=1e-15)
    for i, t in enumerate(rows):
        assert np.allclose(groups[:, i, : t + 1].sum(axis=1), 1.0, atol=1e-12)


def test_per_group_sparse_tables():
    S, Hq, Hkv, d, b, kk = 48, 6, 3, 8, 4, 9
    q, k, v = _qkv(S, Hq, Hkv, d, seed=13)
    rng = np.random.default_rng(14)
    R = (S + b - 1) // b
    shared = np.full((R, kk), -1, dtype=np.int32)
    for r in range(R):
        t1 = min(r * b + b, S) - 1
        m = min(kk, t1 + 1)
        shared[r, :m] = np.sort(rng.choice(t1 + 1, size=m, replace=False))
    # the same table in every group is the shared-support result
    same = np.stack([shared] * Hkv)
    assert np.array_equal(oracle.sparse(q, k, v, same, b), oracle.sparse(q, k, v, shared, b))
    # a head reads only its own group's table
    other = same.copy()
    other[1] = np.roll(shared, 1, axis=1)
    o1, o0 = oracle.sparse(q, k, v, other, b), oracle.sparse(q, k, v, same, b)
    G = Hq // Hkv
    assert np.array_equal(o1[:, :G], o0[:, :G]) and np.array_equal(o1[:, 2 * G:], o0[:, 2 * G:])
    # full per-group budgets reproduce dense attention (fp64 SDPA)
    full = np.stack([np.tile(np.arange(S, dtype=np.int32), (R, 1))] * Hkv)
    qt = torch.from_numpy(q).transpose(0, 1)
    kt = torch.from_numpy(np.repeat(k, G, axis=1)).transpose(0, 1)
    vt = torch.from_numpy(np.repeat(v, G, axis=1)).transpose(0, 1)
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True)
    assert np.allclose(oracle.sparse(q, k, v, full, b), ref.transpose(0, 1).numpy(),
                       rtol=1e-10, atol=1e-12)


# ------------------------------------------------------------ paged K/V cache
def test_paged_cache_matches_contiguous():
    S, Hq, Hkv, d, b, kk, ps = 37, 4, 2, 8, 4, 11, 5
    q, k, v = _qkv(S, Hq, Hkv, d, seed=20)
    rng = np.random.default_rng(21)
    R = (S + b - 1) // b
    idx = np.full((R, kk), -1, dtype=np.int32)
    for r in range(R):
        t1 = min(r * b + b, S) - 1
        m = min(kk, t1 + 1)
        idx[r, :m] = rng.choice(t1 + 1, size=m, replace=False)
    ref = oracle.sparse(q, k, v, idx, b)
    # one page holding everything, identity table
    one = oracle.sparse_paged(q, k[None], v[None], [0], idx, b)
    assert np.array_equal(one, ref)
    # pages scattered over a larger cache through a permuted table
    npg = (S + ps - 1) // ps
    perm = rng.permutation(npg + 3)[:npg]
    kp = np.zeros((npg + 3, ps, Hkv, d))
    vp = np.zeros((npg + 3, ps, Hkv, d))
    for lp in range(npg):
        n = min(ps, S - lp * ps)
        kp[perm[lp], :n] = k[lp * ps: lp * ps + n]
        vp[perm[lp], :n] = v[lp * ps: lp * ps + n]
    assert np.array_equal(oracle.sparse_paged(q, kp, vp, perm, idx, b), ref)
    # a logical page mapped outside the cache: its positions drop out of every support
    bad = perm.copy()
    bad[2] = npg + 3
    dropped = idx.copy()
    dropped[(dropped >= 2 * ps) & (dropped < 3 * ps)] = -1
    assert np.array_equal(oracle.sparse_paged(q, kp, vp, bad, idx, b),
                          oracle.sparse(q, k, v, dropped, b))

"""GPU parity of the NEXT-row entry points against the fp64 oracle.

KL distillation loss (sp_kl_loss). Inputs come from the seeded generators
only; full-size runs are checked on sampled rows.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_07703_amd import binding as B
from synth import make_kl_rows

from helpers import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()


# The kernel sums P (log P - z) and P in fp64 and the exp-sum in fp32 with a
# running max; log and exp are fp32 (relative error a few 1e-7, growing with
# |z - LSE| through the argument rounding). Bounds below leave a 10x margin.
def _check_kl(kl, grad, loss, ref_kl, ref_grad, ref_loss=None):
    ekl = np.abs(kl - ref_kl) - (1e-4 + 1e-5 * np.abs(ref_kl))
    assert np.all(ekl <= 0), f"kl err {np.max(np.abs(kl - ref_kl)):.3e}"
    scale = np.maximum(np.max(np.abs(ref_grad), axis=1, keepdims=True), 1e-30)
    assert np.all(np.abs(grad - ref_grad) <= 1e-5 * scale), \
        f"grad err {np.max(np.abs(grad - ref_grad) / scale):.3e} of row max"
    if ref_loss is not None:
        assert abs(loss - ref_loss) <= 1e-4 + 1e-5 * abs(ref_loss)


@pytest.mark.parametrize("n,S,zero_frac", [(1, 1, 0.0), (50, 300, 0.0), (64, 1000, 0.4),
                                           (7, 33, 0.9)])
def test_kl_loss(n, S, zero_frac):
    say(f"kl n={n} S={S} zero_frac={zero_frac}")
    t = np.random.default_rng(n + S).integers(0, S, size=n)
    t[0] = S - 1
    rows, P, z = make_kl_rows(n, S, seed=n + S, rows=t, zero_frac=zero_frac)
    p = B.Problem(S, 1, 1, 64)
    kl = torch.empty(n, device="cuda")
    loss = torch.empty(1, device="cuda")
    grad = torch.full((n, S), 7.0, device="cuda")
    B.sp_kl_loss(p, rows.cuda(), P.cuda(), z.cuda(), kl, loss, grad)
    torch.cuda.synchronize()
    ref_kl, ref_grad = oracle.kl(P.numpy(), z.numpy(), rows.numpy())
    _check_kl(kl.cpu().double().numpy(), grad.cpu().double().numpy(), loss.item(),
              ref_kl, ref_grad, ref_kl.mean())


def test_kl_loss_long_rows_and_invalid_rows():
    S = 40000   # rows longer than the register-resident limit stream twice
    rows = torch.tensor([S - 1, 32767, 32768, 5, -1, S], dtype=torch.int32)
    _, P, z = make_kl_rows(6, S, seed=3, rows=rows.clamp(0, S - 1), zero_frac=0.1)
    p = B.Problem(S, 1, 1, 64)
    kl = torch.empty(6, device="cuda")
    grad = torch.full((6, S), 7.0, device="cuda")
    B.sp_kl_loss(p, rows.cuda(), P.cuda(), z.cuda(), kl, None, grad)
    torch.cuda.synchronize()
    ref_kl, ref_grad = oracle.kl(P.numpy(), z.numpy(), rows.numpy())
    assert ref_kl[4] == 0.0 and ref_kl[5] == 0.0
    _check_kl(kl.cpu().double().numpy(), grad.cpu().double().numpy(), None, ref_kl, ref_grad)


def test_kl_loss_optional_outputs():
    S, n = 200, 9
    rows, P, z = make_kl_rows(n, S, seed=9)
    p = B.Problem(S, 1, 1, 64)
    rc, Pc, zc = rows.cuda(), P.cuda(), z.cuda()
    grad = torch.empty(n, S, device="cuda")
    B.sp_kl_loss(p, rc, Pc, zc, None, None, grad)          # gradient only
    kl = torch.empty(n, device="cuda")
    B.sp_kl_loss(p, rc, Pc, zc, kl, None, None)            # values only
    torch.cuda.synchronize()
    ref_kl, ref_grad = oracle.kl(P.numpy(), z.numpy(), rows.numpy())
    _check_kl(kl.cpu().double().numpy(), grad.cpu().double().numpy(), None, ref_kl, ref_grad)
    with pytest.raises(B.SparsePrefillError):
        B.sp_kl_loss(p, rc, Pc, zc, None, torch.empty(1, device="cuda"), None)
    B.sp_kl_loss(p, rc[:0], Pc[:0], zc[:0])                 # no rows: a no-op


def test_kl_loss_full_size_sampled():
    S = 32768
    say(f"kl full size S={S}, every query row")
    rows, P, z = make_kl_rows(S, S, seed=4, rows=torch.arange(S), zero_frac=0.2,
                              device="cuda")
    p = B.Problem(S, 1, 1, 64)
    kl = torch.empty(S, device="cuda")
    loss = torch.empty(1, device="cuda")
    grad = torch.empty(S, S, device="cuda")
    B.sp_kl_loss(p, rows, P, z, kl, loss, grad)
    torch.cuda.synchronize()
    sample = np.array([0, 1, 2047, 4096, 16383, 30000, 32766, 32767])
    Ps, zs = P[sample].cpu().numpy(), z[sample].cpu().numpy()
    ref_kl, ref_grad = oracle.kl(Ps, zs, sample)
    # the oracle's gradient is of the mean over its own rows; rescale to S rows
    ref_grad *= len(sample) / S
    _check_kl(kl[sample].cpu().double().numpy(), grad[sample].cpu().double().numpy(), None,
              ref_kl, ref_grad)
    # the mean: fp64 sum of the kernel's own per-row values
    assert loss.item() == pytest.approx(kl.double().mean().item(), rel=1e-6)

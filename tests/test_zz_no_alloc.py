"""The allocation-free fused scoring + top-k (sp_indexer_topk_noalloc) against
the workspace form (sp_indexer_topk), through the C ABI: selections must be
identical (integer output, same kernels). Two calls in a row, the second on
a smaller problem, so the second runs on the static scratch the first left
behind."""
import pytest
import torch

from paper_2606_07703_amd import binding as B
from synth import make_index_vectors

from helpers import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    B.load()


def _pair(S, di, k, W, relu, seed, kind="gauss"):
    say(f"no-alloc fused top-k S={S} d_idx={di} k={k} W={W} relu={relu} {kind}")
    qi, ki = (t.cuda() for t in make_index_vectors(S, di, seed=seed, kind=kind))
    p = B.Problem(S, 1, 1, 64, index_dim=di, topk=k, block_q=1, local_window=W, relu=relu)
    ref = torch.full((S, k), -7, dtype=torch.int32, device="cuda")
    ws = torch.empty(B.sp_workspace_bytes(p, "indexer_topk"), dtype=torch.uint8, device="cuda")
    B.sp_indexer_topk(p, qi, ki, ref, ws)
    got = torch.full((S, k), -7, dtype=torch.int32, device="cuda")
    B.sp_indexer_topk_noalloc(p, qi, ki, got)
    torch.cuda.synchronize()
    same = torch.equal(got, ref)
    say(f"  identical: {same}")
    assert same


def test_noalloc_matches_workspace_form_two_calls():
    _pair(4096, 64, 512, 0, 1, seed=41)
    _pair(1000, 128, 100, 5, 1, seed=42, kind="ternary")


def test_noalloc_rejects_problems_beyond_the_static_scratch():
    S = 30000
    p = B.Problem(S, 1, 1, 64, index_dim=128, topk=64, block_q=1)
    assert B.sp_workspace_bytes(p, "indexer_topk") > (64 << 20)
    qi = torch.zeros(S, 128, dtype=torch.bfloat16, device="cuda")
    idx = torch.empty(S, 64, dtype=torch.int32, device="cuda")
    with pytest.raises(B.SparsePrefillError):
        B.sp_indexer_topk_noalloc(p, qi, qi, idx)

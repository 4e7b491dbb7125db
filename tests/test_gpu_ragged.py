"""GPU parity of the ragged whole-head selection (SA_SELECT_HEAD_TOPK) against
the oracle, bit-exact, and of the scheduled forward on the ragged lists it
produces.  The oracle keeps, per head, every query block's best key block and
then the largest remaining pairs under (score desc, i asc, j asc), with rows
capped at the list stride kmax."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_23153_amd as sa
import workloads as W
from gpu_helpers import check_launch_order, check_out, oracle_attend, say, widen

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TAU = W.softmax_scale(128)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sa.library()
    yield
    torch.cuda.synchronize()


def small_locality(heads=2, grid=(8, 16, 32), seed=5):
    return W.Workload("locality_small", 1, heads, grid, 128, 64, 1000, "locality", seed)


def head_select_and_check(q, k, block, budget, what, kmax=None, heads=None):
    """GPU whole-head selection vs the oracle on every (or the listed) head."""
    B, H, N, _ = q.shape
    nb = O.block_count(N, block)
    width = nb if kmax is None else kmax
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), budget, block=block,
                                     mode=sa.SA_SELECT_HEAD_TOPK, kmax=width)
    torch.cuda.synchronize()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            s = O.block_scores(widen(q[b, h]), widen(k[b, h]), block)
            ri, rc = O.select_head_topk(s, budget=budget, kmax=width)
            assert np.array_equal(cnt_c[b, h], rc), (what, b, h, np.nonzero(cnt_c[b, h] != rc)[0][:5])
            bad = np.nonzero((idx_c[b, h] != ri).any(axis=1))[0]
            assert bad.size == 0, (what, b, h, bad[:5], idx_c[b, h][bad[:1]], ri[bad[:1]])
    say(f"  {what}: head-topk bit-exact, budget {budget} of {nb}x{nb}, "
        f"cnt {int(cnt_c.min())}..{int(cnt_c.max())}")
    return idx, cnt


@pytest.mark.parametrize("block,keep_bp", [(64, 300), (64, 1000), (64, 2500), (128, 1000)])
def test_select_head_locality(block, keep_bp):
    wl = small_locality()
    q, k, _ = W.make_inputs(wl)
    nb = O.block_count(wl.seqlen, block)
    head_select_and_check(q, k, block, O.head_pair_budget(keep_bp, nb, nb),
                          f"locality b={block} keep={keep_bp}")


def test_select_head_normal_ragged_tail():
    g = torch.Generator().manual_seed(21)
    q = torch.randn(2, 3, 1000, 128, generator=g).to(torch.bfloat16)   # 16 blocks, tail 40
    k = torch.randn(2, 3, 1000, 128, generator=g).to(torch.bfloat16)
    head_select_and_check(q, k, 64, O.head_pair_budget(2000, 16, 16), "normal N=1000")


def test_select_head_row_cap():
    wl = small_locality(seed=6)
    q, k, _ = W.make_inputs(wl)
    nb = O.block_count(wl.seqlen, 64)
    for kmax in (1, 3, 9):
        head_select_and_check(q, k, 64, O.head_pair_budget(1500, nb, nb),
                              f"kmax cap {kmax}", kmax=kmax)


def test_select_head_ties():
    # Q = 0: every score ties, so the extra pairs go in (i, j) order
    g = torch.Generator().manual_seed(8)
    k = torch.randn(1, 2, 1000, 128, generator=g).to(torch.bfloat16)
    q = torch.zeros(1, 2, 1000, 128, dtype=torch.bfloat16)
    q[0, 1, :, 3] = -0.0
    for budget in (16, 17, 40, 100, 255, 256):
        head_select_and_check(q, k, 64, budget, f"all-tie budget={budget}")
    # duplicated key blocks: exact ties between pairs of different j
    k2 = torch.randn(1, 1, 1024, 128, generator=g).to(torch.bfloat16)
    k2[0, 0, 512:] = k2[0, 0, :512]
    q2 = torch.randn(1, 1, 1024, 128, generator=g).to(torch.bfloat16)
    for budget in (16, 50, 97):
        head_select_and_check(q2, k2, 64, budget, f"duplicate blocks budget={budget}")


def test_select_head_budget_extremes():
    wl = small_locality(heads=1, seed=7)
    q, k, _ = W.make_inputs(wl)
    nb = O.block_count(wl.seqlen, 64)
    idx, cnt = head_select_and_check(q, k, 64, nb, "budget = nqb (row bests only)")
    assert (cnt.cpu() == 1).all()
    idx, cnt = head_select_and_check(q, k, 64, nb * nb, "budget = all pairs")
    assert (cnt.cpu() == nb).all()


def test_select_head_wan13b():
    wl = W.WORKLOADS["wan13b_480p"]
    q, k, _ = W.make_inputs(wl, heads=[0, 5, 11])
    nb = O.block_count(wl.seqlen, 64)
    head_select_and_check(q, k, 64, O.head_pair_budget(1000, nb, nb), "wan13b_480p")


def test_fwd_on_head_lists():
    wl = small_locality(seed=9)
    q, k, v = W.make_inputs(wl)
    N = wl.seqlen
    for block in (64, 128):
        nb = O.block_count(N, block)
        idx, cnt = head_select_and_check(q, k, block, O.head_pair_budget(1000, nb, nb),
                                         f"fwd lists b={block}")
        order = sa.sparse_attn_schedule(cnt, N, idx.shape[-1], block=block)
        torch.cuda.synchronize()
        check_launch_order(order.cpu().numpy(), cnt.cpu().numpy(), idx.shape[-1], N, block,
                           f"head lists b={block}")
        o, lse = sa.sparse_attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), idx, cnt, block=block,
                                    order=order)
        o0, l0 = sa.sparse_attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), idx, cnt, block=block)
        torch.cuda.synchronize()
        # the launch order changes nothing in the results
        assert torch.equal(o.view(torch.int16), o0.view(torch.int16)) and torch.equal(lse, l0)
        idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
        for h in range(wl.heads):
            ro, rl = oracle_attend(q[0, h], k[0, h], v[0, h], idx_c[0, h], cnt_c[0, h], block, TAU)
            check_out(o[0, h].cpu(), lse[0, h].cpu(), ro, rl, what=f"ragged fwd b={block} h{h}")


@pytest.mark.slow
def test_sweep_full_size_head_topk():
    """The sweep configuration (14B-720P shape, locality inputs) with ragged
    whole-head selection at block 128 / keep 25%: two heads bit-exact, and the
    scheduled forward on 12 sampled query blocks of each."""
    wl = W.WORKLOADS["sweep"]
    heads = [0, wl.heads - 1]
    say("  generating sweep inputs")
    q, k, v = W.make_inputs(wl)
    block, N = 128, wl.seqlen
    nb = O.block_count(N, block)
    budget = O.head_pair_budget(2500, nb, nb)
    idx, cnt = head_select_and_check(q, k, block, budget, "sweep b=128 keep=25%", heads=heads)
    order = sa.sparse_attn_schedule(cnt, N, idx.shape[-1], block=block)
    o, lse = sa.sparse_attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), idx, cnt, block=block,
                                order=order)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    rng = np.random.default_rng(4)
    for h in heads:
        qb = sorted(set(rng.choice(nb - 1, 11, replace=False).tolist()) | {nb - 1})
        ro, rl = oracle_attend(q[0, h], k[0, h], v[0, h], idx_c[0, h], cnt_c[0, h], block, TAU,
                               qblocks=qb)
        rows = np.concatenate([np.arange(i * block, min(i * block + block, N)) for i in qb])
        check_out(o[0, h].cpu(), lse[0, h].cpu(), ro, rl, rows=rows, what=f"sweep fwd h{h}")

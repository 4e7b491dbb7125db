"""GPU parity over the sparsity sweep at the 14B-720P shape (40 heads' worth
of sequence: 75,600 tokens, d = 128; locality inputs with 2% long-range hot
blocks): blocks 64 and 128, keep 3%, 10%, 25% and 100% with the row top-k.
Two heads (0 and 39) are generated and run: selection bit-exact against the
oracle, the scheduled forward against the oracle on sampled query blocks
(the tail block included).  At keep 100% every key block is listed, so the
output is dense attention (the oracle's sparse path at keep 100% is pinned
to dense SDPA on the CPU)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_23153_amd as sa
import workloads as W
from gpu_helpers import check_out, oracle_attend, oracle_select, say

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

DEV = "cuda:0"
TAU = W.softmax_scale(128)
HEADS = (0, 39)


@pytest.fixture(scope="module")
def sweep_inputs():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sa.library()
    wl = W.WORKLOADS["sweep"]
    say("  generating sweep inputs (heads 0, 39)")
    q, k, v = W.make_inputs(wl, heads=HEADS)
    yield wl, (q, k, v), tuple(t.to(DEV) for t in (q, k, v))
    torch.cuda.synchronize()


@pytest.mark.parametrize("block", [64, 128])
@pytest.mark.parametrize("keep_bp", [300, 1000, 2500, 10000])
def test_sweep_point(sweep_inputs, block, keep_bp):
    wl, (q, k, v), (qd, kd, vd) = sweep_inputs
    N = wl.seqlen
    nb = O.block_count(N, block)
    kk = O.keep_count(keep_bp, nb)
    idx, cnt = sa.sparse_attn_select(qd, kd, kk, block=block)
    order = sa.sparse_attn_schedule(cnt, N, kk, block=block)
    o, lse = sa.sparse_attn_fwd(qd, kd, vd, idx, cnt, block=block, order=order)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all() and torch.isfinite(lse).all()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    rng = np.random.default_rng(block + keep_bp)
    nq = 3 if keep_bp == 10000 else 8
    for hi in range(len(HEADS)):
        ri, rc = oracle_select(q[0, hi], k[0, hi], block, keep_bp)
        assert np.array_equal(cnt_c[0, hi], rc), (block, keep_bp, hi)
        bad = np.nonzero((idx_c[0, hi] != ri).any(axis=1))[0]
        assert bad.size == 0, (block, keep_bp, hi, bad[:5])
        if keep_bp == 10000:
            assert np.array_equal(ri, np.tile(np.arange(nb, dtype=ri.dtype), (nb, 1)))
        qb = sorted(set(rng.choice(nb - 1, nq - 1, replace=False).tolist()) | {nb - 1})
        ro, rl = oracle_attend(q[0, hi], k[0, hi], v[0, hi], ri, rc, block, TAU, qblocks=qb)
        rows = np.concatenate([np.arange(i * block, min(i * block + block, N)) for i in qb])
        check_out(o[0, hi].cpu(), lse[0, hi].cpu(), ro, rl, rows=rows,
                  what=f"sweep b={block} keep={keep_bp / 100:g}% h{HEADS[hi]}")
    say(f"  sweep b={block} keep={keep_bp / 100:g}%: k={kk} of {nb}, select bit-exact on "
        f"{len(HEADS)} heads, {nq} query blocks each checked")

"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle on
identical seeded inputs: block index lists bit-exact, bf16 outputs within
rel-L2 1e-2 / max-abs 2e-2."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_23153_amd as sa
import workloads as W
from gpu_helpers import check_launch_order, check_out, oracle_attend, oracle_select, say, widen

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


def to_dev(*ts):
    return [t.to(DEV) for t in ts]


def select_and_check(q, k, block, keep_bp, what):
    """GPU selection of every (b, h) vs the oracle, bit-exact; returns the
    device lists."""
    B, H, N, _ = q.shape
    nb = O.block_count(N, block)
    kk = O.keep_count(keep_bp, nb)
    qd, kd = to_dev(q, k)
    idx, cnt = sa.sparse_attn_select(qd, kd, kk, block=block)
    torch.cuda.synchronize()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    for b in range(B):
        for h in range(H):
            ri, rc = oracle_select(q[b, h], k[b, h], block, keep_bp)
            assert np.array_equal(cnt_c[b, h], rc), (what, b, h)
            bad = np.nonzero((idx_c[b, h] != ri).any(axis=1))[0]
            assert bad.size == 0, (what, b, h, bad[:5], idx_c[b, h][bad[:1]], ri[bad[:1]])
    say(f"  {what}: select bit-exact over {B * H} heads (k={kk} of {nb})")
    return idx, cnt


# ------------------------------------------------------------------ select
def test_select_tiny_bitexact():
    wl = W.WORKLOADS["tiny"]
    q, k, _ = W.make_inputs(wl)
    select_and_check(q, k, wl.block, wl.keep_bp, "tiny")


def test_select_wan13b_bitexact():
    wl = W.WORKLOADS["wan13b_480p"]
    q, k, _ = W.make_inputs(wl)
    select_and_check(q, k, wl.block, wl.keep_bp, "wan13b_480p")


def test_select_ties_and_signed_zeros():
    # Q = 0: every score is +-0, so each row keeps blocks 0..k-1.
    N = 1000  # 16 blocks, tail of 40
    g = torch.Generator().manual_seed(5)
    k = torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16)
    q = torch.zeros(1, 2, N, 128, dtype=torch.bfloat16)
    q[0, 1, :, 0] = -0.0
    idx, cnt = select_and_check(q, k, 64, 2500, "zero-q ties")
    assert (idx.cpu()[..., :4] == torch.arange(4, dtype=torch.int32)).all()
    # duplicated key blocks give exact ties between different indices
    k2 = torch.randn(1, 1, 512, 128, generator=g).to(torch.bfloat16)
    k2[0, 0, 256:] = k2[0, 0, :256]
    q2 = torch.randn(1, 1, 512, 128, generator=g).to(torch.bfloat16)
    select_and_check(q2, k2, 64, 5000, "duplicate-block ties")


def test_select_low_word_ties():
    """Block scores that agree in the high 32 bits of their fp64 order keys
    and differ only in the low bits (relative gaps ~4e-9), with exact ties
    among them: the top-k must still follow the full fp64 order."""
    nb, block = 16, 64
    q = torch.zeros(1, 1, nb * block, 128)
    q[..., 0] = 1.0                          # score_ij = mean of k[:, 0] over block j
    k = torch.zeros(1, 1, nb * block, 128)
    k[0, 0, :, 0] = 2.0 ** 14
    for j in range(nb):
        rank = (7 * j) % nb // 2             # pairs of blocks share a rank: exact ties
        k[0, 0, j * block, 0] = rank * 2.0 ** -8
    q, k = q.to(torch.bfloat16), k.to(torch.bfloat16)
    for keep in (1000, 2500, 5000, 7000):
        select_and_check(q, k, block, keep, f"low-word ties keep={keep}")


@pytest.mark.parametrize("N,block,keep_bp", [(4096, 128, 1000), (777, 64, 3000),
                                             (64, 64, 100), (8200, 128, 10000)])
def test_select_shapes(N, block, keep_bp):
    g = torch.Generator().manual_seed(N + block)
    q = torch.randn(2, 3, N, 128, generator=g).to(torch.bfloat16)
    k = torch.randn(2, 3, N, 128, generator=g).to(torch.bfloat16)
    select_and_check(q, k, block, keep_bp, f"N={N} b={block} keep={keep_bp}")


def test_select_wan14b_low_locality_all_heads():
    """The 14B-720P layer with i.i.d. normal Q and K: pooled scores with much
    cancellation, so many rows have a k-th gap within the approximation's
    bound; every head bit-exact."""
    wl = W.WORKLOADS["wan14b_720p_normal"]
    say("  generating wan14b_720p_normal inputs")
    q, k, _ = W.make_inputs(wl)
    select_and_check(q, k, wl.block, wl.keep_bp, "wan14b normal")


def test_select_ties_beyond_one_wave():
    """Q = 0 over 128 key blocks: every score is 0 and more than 64 blocks tie
    at the k-th place.  Then keys that repeat every 64 blocks: each score
    appears 4 times, and k not a multiple of 4 splits a tied group."""
    g = torch.Generator().manual_seed(11)
    N = 128 * 64
    k = torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16)
    q = torch.zeros(1, 2, N, 128, dtype=torch.bfloat16)
    idx, _ = select_and_check(q, k, 64, 1000, "zero-q over 128 blocks")
    assert (idx.cpu()[..., :13] == torch.arange(13, dtype=torch.int32)).all()
    k2 = torch.randn(1, 2, 64 * 64, 128, generator=g).to(torch.bfloat16).repeat(1, 1, 4, 1)
    q2 = torch.randn(1, 2, 256 * 64, 128, generator=g).to(torch.bfloat16)
    for keep in (350, 1000):  # k = 9, 26
        select_and_check(q2, k2, 64, keep, f"period-64 key blocks keep={keep}")


@pytest.mark.parametrize("qexp,kexp", [(60, 0), (-100, 0), (50, 50)])
def test_select_extreme_magnitudes(qexp, kexp):
    """Inputs scaled by powers of two: pooled norms beyond the approximation's
    range (2^60, rescored exactly), near the fp32 flush range, and large on
    both sides.  Scaling by a power of two does not change the ranking."""
    g = torch.Generator().manual_seed(200 + qexp)
    N = 200 * 64 - 5
    q = (torch.randn(1, 2, N, 128, generator=g) * 2.0 ** qexp).to(torch.bfloat16)
    k = (torch.randn(1, 2, N, 128, generator=g) * 2.0 ** kexp).to(torch.bfloat16)
    select_and_check(q, k, 64, 300, f"q*2^{qexp} k*2^{kexp}")


@pytest.mark.parametrize("nb", [584, 585, 1192, 1193])
def test_select_on_chip_capacity_edges(nb):
    """Around the on-chip score rows: 584 blocks (two workgroups per CU), 585
    and 1192 (one), 1193 (the fp64 score matrix in the workspace)."""
    g = torch.Generator().manual_seed(nb)
    N = nb * 64 - 17
    q = torch.randn(1, 1, N, 128, generator=g).to(torch.bfloat16)
    k = torch.randn(1, 1, N, 128, generator=g).to(torch.bfloat16)
    select_and_check(q, k, 64, 300, f"nb={nb}")


@pytest.mark.parametrize("N,block", [(4160, 128), (1000, 64)])
def test_select_token_major_batched(N, block):
    """Token-major [B, L, H, d] views with two batches: the fused kernel's
    in-kernel query pooling and the key pooling address every (b, h) through
    the strides; lists bit-exact, including the ragged last block."""
    g = torch.Generator().manual_seed(7 * N + block)
    base = [torch.randn(2, N, 3, 128, generator=g).to(torch.bfloat16) for _ in range(2)]
    q, k = (t.permute(0, 2, 1, 3) for t in base)
    select_and_check(q, k, block, 1000, f"token-major B=2 N={N} b={block}")


def test_select_kmax_padding():
    g = torch.Generator().manual_seed(3)
    q = torch.randn(1, 1, 2048, 128, generator=g).to(torch.bfloat16)
    k = torch.randn(1, 1, 2048, 128, generator=g).to(torch.bfloat16)
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), 5, kmax=9)
    idx = idx.cpu()
    ri, _ = oracle_select(q[0, 0], k[0, 0], 64, 1500)
    assert (cnt.cpu() == 5).all()
    assert np.array_equal(idx[0, 0, :, :5].numpy(), ri)
    assert (idx[..., 5:] == -1).all()


# --------------------------------------------------------------------- fwd
def fwd_and_check(q, k, v, idx, cnt, block, what, qblocks=None, heads=None, schedule=True):
    qd, kd, vd = to_dev(q, k, v)
    order = None
    if schedule:
        order = sa.sparse_attn_schedule(cnt, q.shape[2], idx.shape[-1], block=block)
        torch.cuda.synchronize()
        check_launch_order(order.cpu().numpy(), cnt.cpu().numpy(), idx.shape[-1], q.shape[2],
                           block, what)
    o, lse = sa.sparse_attn_fwd(qd, kd, vd, idx, cnt, block=block, order=order)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    B, H, N, _ = q.shape
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            ro, rl = oracle_attend(q[b, h], k[b, h], v[b, h], idx_c[b, h], cnt_c[b, h], block,
                                   TAU, qblocks)
            rows = None
            if qblocks is not None:
                rows = np.concatenate([np.arange(i * block, min(i * block + block, N))
                                       for i in qblocks])
            check_out(o[b, h], lse[b, h], ro, rl, rows=rows, what=f"{what} b{b} h{h}")
    return o, lse


@pytest.mark.parametrize("schedule", [True, False])
def test_fwd_tiny(schedule):
    wl = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(wl)
    idx, cnt = select_and_check(q, k, wl.block, wl.keep_bp, "tiny")
    fwd_and_check(q, k, v, idx, cnt, wl.block, "tiny fwd", schedule=schedule)


def test_schedule_large_ragged_properties():
    # 3 x 40 heads x 1182 blocks of ragged lengths: several XCD groups and a
    # partial tail group; the order is a permutation whose sorted positions
    # carry non-increasing cost classes, raster order within a class
    rng = np.random.default_rng(21)
    cnt = rng.integers(0, 300, size=(3, 40, 1182)).astype(np.int32)
    cnt[0, 0, :50] = 0
    cntd = torch.from_numpy(cnt).to(DEV)
    order = sa.sparse_attn_schedule(cntd, 75600, 250, block=64)
    torch.cuda.synchronize()
    check_launch_order(order.cpu().numpy(), cnt, 250, 75600, 64, "ragged b64")
    order = sa.sparse_attn_schedule(cntd[:, :, :591].contiguous(), 75600, 250, block=128)
    with pytest.raises(ValueError):
        sa.sparse_attn_schedule(cntd[:, :, :591], 75600, 250, block=128)
    torch.cuda.synchronize()
    check_launch_order(order.cpu().numpy(), cnt[:, :, :591], 250, 75600, 128, "ragged b128")
    # uniform lists: one class, so the order is the XCD interleave of raster order
    cnt1 = np.full((1, 40, 1182), 36, dtype=np.int32)
    order = sa.sparse_attn_schedule(torch.from_numpy(cnt1).to(DEV), 75600, 36, block=64)
    torch.cuda.synchronize()
    check_launch_order(order.cpu().numpy(), cnt1, 36, 75600, 64, "uniform")


def test_fwd_wan13b_sampled_heads():
    wl = W.WORKLOADS["wan13b_480p"]
    q, k, v = W.make_inputs(wl)
    idx, cnt = select_and_check(q, k, wl.block, wl.keep_bp, "wan13b_480p")
    fwd_and_check(q, k, v, idx, cnt, wl.block, "wan13b fwd", heads=[0, 5, 11])


@pytest.mark.parametrize("N,block", [(1000, 64), (1000, 128), (4096, 128), (200, 64)])
def test_fwd_ragged_lists_with_empty_rows(N, block):
    g = torch.Generator().manual_seed(N * 7 + block)
    q = torch.randn(2, 2, N, 128, generator=g).to(torch.bfloat16)
    k = torch.randn(2, 2, N, 128, generator=g).to(torch.bfloat16)
    v = torch.randn(2, 2, N, 128, generator=g).to(torch.bfloat16)
    nb = O.block_count(N, block)
    kmax = min(nb, 9)
    idx = np.full((2, 2, nb, kmax + 2), -1, dtype=np.int32)
    cnt = np.zeros((2, 2, nb), dtype=np.int32)
    for b in range(2):
        for h in range(2):
            ii, cc = W.random_block_lists(nb, nb, kmax, seed=100 * b + h + N, p_empty=0.15)
            idx[b, h, :, :kmax], cnt[b, h] = ii, cc
    fwd_and_check(q, k, v, torch.from_numpy(idx).to(DEV), torch.from_numpy(cnt).to(DEV), block,
                  f"ragged N={N} b={block}")


def test_fwd_keep_all_is_dense():
    g = torch.Generator().manual_seed(11)
    N = 700
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    idx, cnt = select_and_check(q, k, 64, 10000, "dense select")
    o, _ = fwd_and_check(q, k, v, idx, cnt, 64, "dense fwd")
    ref = torch.nn.functional.scaled_dot_product_attention(
        q.to(torch.float64), k.to(torch.float64), v.to(torch.float64), scale=TAU)
    assert (o.to(torch.float64) - ref).abs().max() < 2e-2


def test_fwd_strided_token_major_layout():
    # [B, N, H, d] storage viewed as [B, H, N, d]: strides (N*H*d, d, H*d)
    g = torch.Generator().manual_seed(12)
    N, H = 1500, 3
    base = [torch.randn(1, N, H, 128, generator=g).to(torch.bfloat16) for _ in range(3)]
    q, k, v = (t.permute(0, 2, 1, 3) for t in base)
    idx, cnt = select_and_check(q, k, 64, 2000, "strided select")
    qd, kd, vd = (t.to(DEV).permute(0, 2, 1, 3) for t in base)
    o = torch.empty(1, N, H, 128, dtype=torch.bfloat16, device=DEV).permute(0, 2, 1, 3)
    o, lse = sa.sparse_attn_fwd(qd, kd, vd, idx, cnt, o=o)
    torch.cuda.synchronize()
    for h in range(H):
        ro, rl = oracle_attend(q[0, h], k[0, h], v[0, h], idx.cpu().numpy()[0, h],
                               cnt.cpu().numpy()[0, h], 64, TAU)
        check_out(o[0, h].cpu(), lse[0, h].cpu(), ro, rl, what=f"strided h{h}")


def test_fwd_is_deterministic():
    wl = W.WORKLOADS["tiny"]
    q, k, v = to_dev(*W.make_inputs(wl))
    idx, cnt = sa.sparse_attn_select(q, k, 7)
    o1, l1 = sa.sparse_attn_fwd(q, k, v, idx, cnt)
    o2, l2 = sa.sparse_attn_fwd(q, k, v, idx, cnt)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.slow
def test_wan14b_full_size_sampled():
    """Full 40-head 75,600-token layer at 97% sparsity, in the launch
    configuration the benchmark times; the oracle checks the selection of
    all 40 heads and, in heads 0 and 39, 20 query blocks (including the
    16-token tail block) of the output."""
    wl = W.WORKLOADS["wan14b_720p"]
    say("  generating wan14b_720p inputs")
    q, k, v = W.make_inputs(wl)
    qd, kd, vd = to_dev(q, k, v)
    nb = O.block_count(wl.seqlen, wl.block)
    kk = O.keep_count(wl.keep_bp, nb)
    idx, cnt = sa.sparse_attn_select(qd, kd, kk)
    order = sa.sparse_attn_schedule(cnt, wl.seqlen, kk)
    o, lse = sa.sparse_attn_fwd(qd, kd, vd, idx, cnt, order=order)
    torch.cuda.synchronize()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    rng = np.random.default_rng(14)
    for h in range(wl.heads):  # selection: every head
        ri, rc = oracle_select(q[0, h], k[0, h], wl.block, wl.keep_bp)
        assert np.array_equal(idx_c[0, h], ri) and np.array_equal(cnt_c[0, h], rc), h
        if h not in (0, 39):
            continue
        qb = sorted(set(rng.choice(nb - 1, 19, replace=False).tolist()) | {nb - 1})
        res = O.sparse_attention(widen(q[0, h]), widen(k[0, h]), widen(v[0, h]), ri, rc,
                                 wl.block, TAU, qblocks=qb)
        rows = np.concatenate([np.arange(i * 64, min(i * 64 + 64, wl.seqlen)) for i in qb])
        check_out(o[0, h].cpu(), lse[0, h].cpu(), res[0], res[1], rows=rows,
                  what=f"wan14b h{h}")
    # property at any size: every output row is finite and LSE finite
    assert torch.isfinite(o).all() and torch.isfinite(lse).all()
    # raster order (no schedule) gives the same bits
    o0, l0 = sa.sparse_attn_fwd(qd, kd, vd, idx, cnt)
    torch.cuda.synchronize()
    assert torch.equal(o0.cpu().view(torch.int16), o.cpu().view(torch.int16))
    assert torch.equal(l0.cpu().view(torch.int32), lse.cpu().view(torch.int32))
    check_launch_order(order.cpu().numpy(), cnt_c, kk, wl.seqlen, wl.block, "wan14b")


# ---------------------------------------------------- block-128 tail blocks
def tail_lists(nb, kmax, seed, B=1, H=2):
    """Random ragged lists (about 10% empty) in which a third of the rows
    list the last key block, so the tail block is walked often."""
    idx = np.full((B, H, nb, kmax), -1, dtype=np.int32)
    cnt = np.zeros((B, H, nb), dtype=np.int32)
    for b in range(B):
        for h in range(H):
            ii, cc = W.random_block_lists(nb, nb, kmax, seed=seed + 10 * b + h, p_empty=0.1)
            for i in range(0, nb, 3):
                if cc[i] > 0 and nb - 1 not in ii[i, :cc[i]]:
                    ii[i, cc[i] - 1] = nb - 1
                    ii[i, :cc[i]] = np.sort(ii[i, :cc[i]])
            idx[b, h], cnt[b, h] = ii, cc
    return torch.from_numpy(idx), torch.from_numpy(cnt)


@pytest.mark.parametrize("N", [1064, 4160, 8200])
def test_fwd_block128_tail_sub_tile_past_end(N):
    """Block 128 with N mod 128 in (0, 64]: the last block's second 64-row
    sub-tile lies wholly past N (as query tile and as key tile), so the tile
    cursors skip it; tails of 40, 64 and 8 tokens."""
    assert 0 < N % 128 <= 64
    g = torch.Generator().manual_seed(N)
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    nb = O.block_count(N, 128)
    idx, cnt = tail_lists(nb, min(nb, 7), seed=N)
    idx, cnt = idx.to(DEV), cnt.to(DEV)
    for sched in (True, False):
        fwd_and_check(q, k, v, idx, cnt, 128, f"b128 tail N={N} sched={sched}", schedule=sched)


@pytest.mark.parametrize("N,block", [(1000, 64), (4160, 128), (3000, 64)])
def test_fwd_order_does_not_change_results(N, block):
    """The launch order only moves work between CUs: outputs and LSE with the
    scheduled order and with raster order (order = NULL) are the same bits,
    on ragged lists with empty rows and a tail block."""
    g = torch.Generator().manual_seed(N + 3 * block)
    q, k, v = (torch.randn(2, 3, N, 128, generator=g).to(torch.bfloat16).to(DEV)
               for _ in range(3))
    nb = O.block_count(N, block)
    idx, cnt = tail_lists(nb, min(nb, 9), seed=N + 1, B=2, H=3)
    idx, cnt = idx.to(DEV), cnt.to(DEV)
    order = sa.sparse_attn_schedule(cnt, N, idx.shape[-1], block=block)
    o1, l1 = sa.sparse_attn_fwd(q, k, v, idx, cnt, block=block, order=order)
    o0, l0 = sa.sparse_attn_fwd(q, k, v, idx, cnt, block=block)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o0.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l0.view(torch.int32))

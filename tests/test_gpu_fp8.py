"""GPU parity of the fp8 path against the fp64 oracle: e4m3 quantisation
bit-exact (codes and power-of-two block scales), and the fp8 sparse forward
within rel-L2 5e-2 of the oracle run on the oracle's dequantised operands.
Selection always runs on the bf16 inputs."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_23153_amd as sa
import workloads as W
from gpu_helpers import (FP8_LSE_ABS, FP8_REL_L2, check_out, fp8_tiles_to_rows, oracle_select,
                         rel_l2, say, widen)

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


def quant_operands(qd, kd, vd, block):
    """Q row-major, K and V in the fp8 forward's tile layouts."""
    q8, sq = sa.sparse_attn_quant_fp8(qd, block=block)
    k8, sk = sa.sparse_attn_quant_fp8_tiles(kd, sa.SA_FP8_K, block=block)
    v8, sv = sa.sparse_attn_quant_fp8_tiles(vd, sa.SA_FP8_V, block=block)
    return q8, sq, k8, sk, v8, sv


def quant_check(x, block, what, operand=None):
    """GPU quantisation of x [B, H, N, 128] bf16 vs the oracle, bit-exact;
    operand None: the row-major call, else the tile layout of that operand
    (read back through its inverse, and every code past N zero)."""
    B, H, N, _ = x.shape
    if operand is None:
        x8, sc = sa.sparse_attn_quant_fp8(x.to(DEV), block=block)
    else:
        x8t = torch.full((B, H, -(-N // 64), 8192), 0x5A, dtype=torch.uint8, device=DEV)
        x8, sc = sa.sparse_attn_quant_fp8_tiles(x.to(DEV), operand, block=block, x8=x8t)
    torch.cuda.synchronize()
    x8, sc = x8.cpu().numpy(), sc.cpu().numpy()
    if operand is not None:
        x8, pad = fp8_tiles_to_rows(x8, N, operand)
        assert (pad == 0).all(), (what, "codes past N")
    for b in range(B):
        for h in range(H):
            codes, scales = O.quantize_fp8_blocks(widen(x[b, h]), block)
            assert np.array_equal(sc[b, h], scales.astype(np.float32)), (what, b, h)
            bad = np.argwhere(x8[b, h] != codes)
            assert bad.size == 0, (what, b, h, bad[:3], x8[b, h][tuple(bad[0])],
                                   codes[tuple(bad[0])])
    say(f"  {what}: quant bit-exact over {B * H} heads")
    return x8, sc


@pytest.mark.parametrize("N,block", [(4096, 64), (1000, 64), (1000, 128), (77, 64)])
def test_quant_fp8_bitexact(N, block):
    g = torch.Generator().manual_seed(N + block)
    x = torch.randn(2, 3, N, 128, generator=g) * 3
    x[0, 0, :block] = 0.0                                   # all-zero block -> scale 1
    x[0, 1, :block] *= 1000.0                               # large block
    x[0, 2, :block] *= 1e-30                                # tiny block
    x[1, 0, :block] = -0.0                                  # negative zeros
    x[1, 1, 5, 7] = 448.0 * 2.0 ** -3                       # amax exactly 448 * 2^e
    x[1, 2, block:2 * block] = torch.round(x[1, 2, block:2 * block] * 4) / 4  # many ties
    xb = x.to(torch.bfloat16)
    quant_check(xb, block, f"N={N} b={block}")
    quant_check(xb, block, f"N={N} b={block} K tiles", operand=sa.SA_FP8_K)
    quant_check(xb, block, f"N={N} b={block} V tiles", operand=sa.SA_FP8_V)


@pytest.mark.parametrize("N,block", [(4160, 128), (8200, 128), (64, 64), (65, 64)])
def test_quant_fp8_tiles_tails(N, block):
    """Tile layouts where the last 64-key tile is partial or (block 128,
    N mod 128 in (0, 64]) the block's second tile lies past N."""
    g = torch.Generator().manual_seed(7 * N + block)
    x = (torch.randn(1, 2, N, 128, generator=g) * 2).to(torch.bfloat16)
    for op, name in ((sa.SA_FP8_K, "K"), (sa.SA_FP8_V, "V")):
        quant_check(x, block, f"N={N} b={block} {name} tiles", operand=op)


@pytest.mark.parametrize("N,block", [(1000, 64), (4160, 128)])
def test_quant_fp8_token_major(N, block):
    """Token-major [B, L, H, d] views (strides (L H d, d, H d)): all three
    quantisation layouts bit-exact, the strides taken from the view."""
    g = torch.Generator().manual_seed(3 * N + block)
    x = (torch.randn(2, N, 3, 128, generator=g) * 2).to(torch.bfloat16).permute(0, 2, 1, 3)
    quant_check(x, block, f"token-major N={N} b={block}")
    for op, name in ((sa.SA_FP8_K, "K"), (sa.SA_FP8_V, "V")):
        quant_check(x, block, f"token-major N={N} b={block} {name} tiles", operand=op)


def test_quant_fp8_outlier_workload_heads():
    wl = W.WORKLOADS["wan14b_720p_fp8"]
    heads = sorted({h for h, _ in W._outlier_pairs(wl)[0]} | {0})[:3]
    q, k, v = W.make_inputs(wl, heads=heads)
    for name, t, op in (("q", q, None), ("k", k, sa.SA_FP8_K), ("v", v, sa.SA_FP8_V)):
        quant_check(t, wl.block, f"wan14b_720p_fp8 {name} heads {heads}", operand=op)


def fp8_fwd_and_check(q, k, v, idx, cnt, block, what, rows_of=None):
    """Quantise on the GPU, run the fp8 forward, compare with the oracle on
    the oracle's own dequantised operands."""
    qd, kd, vd = (t.to(DEV) for t in (q, k, v))
    q8, sq, k8, sk, v8, sv = quant_operands(qd, kd, vd, block)
    order = sa.sparse_attn_schedule(cnt, q.shape[2], idx.shape[-1], block=block)
    o, lse = sa.sparse_attn_fwd_fp8(q8, sq, k8, sk, v8, sv, idx, cnt, block=block, order=order)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    B, H, N, _ = q.shape
    worst = 0.0
    for b in range(B):
        for h in range(H):
            deq = [O.dequantize_fp8_blocks(*O.quantize_fp8_blocks(widen(t[b, h]), block), block)
                   for t in (q, k, v)]
            qblocks = None if rows_of is None else rows_of
            ro, rl = O.sparse_attention(*deq, idx_c[b, h], cnt_c[b, h], block, TAU, qblocks)
            rows = None
            if qblocks is not None:
                rows = np.concatenate([np.arange(i * block, min(i * block + block, N))
                                       for i in qblocks])
            check_out(o[b, h], None, ro, rl, rows=rows, rel=FP8_REL_L2, mabs=None,
                      what=f"{what} b{b} h{h}")
            got = o[b, h].to(torch.float64).numpy()
            ref32 = O.sparse_attention(widen(q[b, h]), widen(k[b, h]), widen(v[b, h]),
                                       idx_c[b, h], cnt_c[b, h], block, TAU, qblocks)[0]
            sel = slice(None) if rows is None else rows
            worst = max(worst, rel_l2(got[sel], ref32[sel]))
            fin = np.isfinite(rl) if rows is None else np.isfinite(rl[rows])
            lg = lse[b, h].numpy() if rows is None else lse[b, h].numpy()[rows]
            lr = rl if rows is None else rl[rows]
            assert np.array_equal(np.isneginf(lg), np.isneginf(lr))
            assert np.abs(lg[fin] - lr[fin]).max() <= FP8_LSE_ABS
    say(f"  {what}: rel-L2 vs unquantised bf16 oracle (information) {worst:.3e}")
    return o


def test_fwd_fp8_tiny():
    wl = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(wl)
    kk = O.keep_count(wl.keep_bp, 64)
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), kk)
    fp8_fwd_and_check(q, k, v, idx, cnt, 64, "tiny fp8")


@pytest.mark.parametrize("N,block", [(1000, 64), (1000, 128), (4096, 128), (130, 64)])
def test_fwd_fp8_ragged_lists(N, block):
    g = torch.Generator().manual_seed(N * 3 + block)
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    nb = O.block_count(N, block)
    kmax = min(nb, 7)
    idx = np.full((1, 2, nb, kmax + 1), -1, dtype=np.int32)
    cnt = np.zeros((1, 2, nb), dtype=np.int32)
    for h in range(2):
        ii, cc = W.random_block_lists(nb, nb, kmax, seed=N + h, p_empty=0.15)
        idx[0, h, :, :kmax], cnt[0, h] = ii, cc
    fp8_fwd_and_check(q, k, v, torch.from_numpy(idx).to(DEV), torch.from_numpy(cnt).to(DEV),
                      block, f"fp8 ragged N={N} b={block}")


def test_fwd_fp8_wan13b_sampled():
    wl = W.WORKLOADS["wan13b_480p"]
    q, k, v = W.make_inputs(wl, heads=[0, 7])
    kk = O.keep_count(wl.keep_bp, 512)
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), kk)
    fp8_fwd_and_check(q, k, v, idx, cnt, 64, "wan13b fp8", rows_of=list(range(0, 512, 16)) + [511])


@pytest.mark.slow
def test_wan14b_fp8_full_size_sampled():
    """Full 40-head fp8 layer with channel outliers; oracle on two heads
    (one carrying outliers) at 16 sampled query blocks each."""
    wl = W.WORKLOADS["wan14b_720p_fp8"]
    say("  generating wan14b_720p_fp8 inputs")
    q, k, v = W.make_inputs(wl)
    qd, kd, vd = (t.to(DEV) for t in (q, k, v))
    nb = O.block_count(wl.seqlen, wl.block)
    kk = O.keep_count(wl.keep_bp, nb)
    idx, cnt = sa.sparse_attn_select(qd, kd, kk)
    q8, sq, k8, sk, v8, sv = quant_operands(qd, kd, vd, 64)
    order = sa.sparse_attn_schedule(cnt, wl.seqlen, kk)
    o, lse = sa.sparse_attn_fwd_fp8(q8, sq, k8, sk, v8, sv, idx, cnt, order=order)
    o0, l0 = sa.sparse_attn_fwd_fp8(q8, sq, k8, sk, v8, sv, idx, cnt)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all() and torch.isfinite(lse).all()
    # raster order (no schedule) gives the same bits
    assert torch.equal(o0.view(torch.int16), o.view(torch.int16))
    assert torch.equal(l0.view(torch.int32), lse.view(torch.int32))
    del o0, l0
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    out_head = W._outlier_pairs(wl)[0][0][0]
    rng = np.random.default_rng(3)
    for h in sorted({0, out_head}):
        ri, rc = oracle_select(q[0, h], k[0, h], wl.block, wl.keep_bp)
        assert np.array_equal(idx_c[0, h], ri)
        deq = [O.dequantize_fp8_blocks(*O.quantize_fp8_blocks(widen(t[0, h]), 64), 64)
               for t in (q, k, v)]
        qb = sorted(set(rng.choice(nb - 1, 15, replace=False).tolist()) | {nb - 1})
        ro, rl = O.sparse_attention(*deq, ri, rc, 64, TAU, qblocks=qb)
        rows = np.concatenate([np.arange(i * 64, min(i * 64 + 64, wl.seqlen)) for i in qb])
        check_out(o[0, h].cpu(), None, ro, rl, rows=rows, rel=FP8_REL_L2, mabs=None,
                  what=f"wan14b fp8 h{h}")


@pytest.mark.parametrize("N", [1064, 4160, 8200])
def test_fwd_fp8_block128_tail_sub_tile_past_end(N):
    """Block 128 with N mod 128 in (0, 64]: the last block's second 64-token
    sub-tile lies wholly past N (skipped by the pair cursor as key tile, and
    a query tile with no rows); lists often include the tail block."""
    from test_gpu_parity import tail_lists
    g = torch.Generator().manual_seed(N + 5)
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    nb = O.block_count(N, 128)
    idx, cnt = tail_lists(nb, min(nb, 7), seed=N + 2)
    fp8_fwd_and_check(q, k, v, idx.to(DEV), cnt.to(DEV), 128, f"fp8 b128 tail N={N}")


@pytest.mark.parametrize("N,block", [(1000, 64), (4160, 128)])
def test_fwd_fp8_order_does_not_change_results(N, block):
    from test_gpu_parity import tail_lists
    g = torch.Generator().manual_seed(N + 7 * block)
    x = [torch.randn(2, 3, N, 128, generator=g).to(torch.bfloat16).to(DEV) for _ in range(3)]
    q8, sq, k8, sk, v8, sv = quant_operands(x[0], x[1], x[2], block)
    nb = O.block_count(N, block)
    idx, cnt = tail_lists(nb, min(nb, 9), seed=N + 3, B=2, H=3)
    idx, cnt = idx.to(DEV), cnt.to(DEV)
    order = sa.sparse_attn_schedule(cnt, N, idx.shape[-1], block=block)
    o1, l1 = sa.sparse_attn_fwd_fp8(q8, sq, k8, sk, v8, sv, idx, cnt, block=block, order=order)
    o0, l0 = sa.sparse_attn_fwd_fp8(q8, sq, k8, sk, v8, sv, idx, cnt, block=block)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o0.view(torch.int16))
    assert torch.equal(l1.view(torch.int32), l0.view(torch.int32))

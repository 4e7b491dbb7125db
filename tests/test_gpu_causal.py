"""GPU parity of the causal-window restriction (paper §1, the sparse branch
restricted to a causal window for auto-regressive generation) through the C
ABI against the fp64 oracle on identical seeded inputs: candidate-restricted
index lists and counts bit-exact, bf16 outputs within rel-L2 1e-2 / max-abs
2e-2, fp8 outputs within rel-L2 5e-2, rows left without allowed keys O = 0
and LSE = -inf."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_23153_amd as sa
import workloads as W
from gpu_helpers import FP8_REL_L2, check_out, say, widen

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


def select_causal_check(q, k, block, keep_bp, causal, what, heads=None):
    B, H, N, _ = q.shape
    nb = O.block_count(N, block)
    kk = O.keep_count(keep_bp, nb)
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), kk, block=block, causal=causal)
    torch.cuda.synchronize()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            ri, rc = O.select_causal(widen(q[b, h]), widen(k[b, h]), block, keep_bp, *causal)
            assert np.array_equal(cnt_c[b, h], rc), (what, b, h)
            bad = np.nonzero((idx_c[b, h] != ri).any(axis=1))[0]
            assert bad.size == 0, (what, b, h, bad[:5])
    say(f"  {what}: causal select bit-exact (k={kk} of {nb}, counts "
        f"{int(cnt_c.min())}..{int(cnt_c.max())})")
    return idx, cnt


def fwd_causal_check(q, k, v, idx, cnt, block, causal, what, heads=None, qblocks=None):
    B, H, N, _ = q.shape
    order = sa.sparse_attn_schedule(cnt, N, idx.shape[-1], block=block)
    o, lse = sa.sparse_attn_fwd(q.to(DEV), k.to(DEV), v.to(DEV), idx, cnt, block=block,
                                order=order, causal=causal)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            ro, rl = O.sparse_attention_causal(widen(q[b, h]), widen(k[b, h]), widen(v[b, h]),
                                               idx_c[b, h], cnt_c[b, h], block, TAU, *causal,
                                               qblocks=qblocks)
            rows = None
            if qblocks is not None:
                rows = np.concatenate([np.arange(i * block, min(i * block + block, N))
                                       for i in qblocks])
            check_out(o[b, h], lse[b, h], ro, rl, rows=rows, what=f"{what} b{b} h{h}")
    return o, lse


@pytest.mark.parametrize("causal", [(1024, 0), (1024, 2), (2048, 1)])
def test_causal_tiny(causal):
    """4 frames of 32 x 32 tokens, chunks of 1 or 2 frames."""
    wl = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(wl)
    idx, cnt = select_causal_check(q, k, wl.block, wl.keep_bp, causal, f"tiny {causal}")
    fwd_causal_check(q, k, v, idx, cnt, wl.block, causal, f"tiny fwd {causal}")


@pytest.mark.parametrize("N,block,causal,keep_bp", [(1000, 64, (600, 1), 1500),
                                                    (1000, 128, (300, 0), 1500),
                                                    (3000, 64, (1000, 2), 1500),
                                                    (777, 64, (777, 0), 1500),
                                                    (1000, 64, (150, 1), 5000)])
def test_causal_unaligned_chunks(N, block, causal, keep_bp):
    """Chunk boundaries inside blocks and a ragged last block; the last case
    keeps 8 of 16 blocks but has only 2 to 6 candidates per query block, so
    the counts fall below k."""
    g = torch.Generator().manual_seed(N + block + causal[0])
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    idx, cnt = select_causal_check(q, k, block, keep_bp, causal, f"N={N} b={block} {causal}")
    fwd_causal_check(q, k, v, idx, cnt, block, causal, f"N={N} b={block} {causal} fwd")


def test_causal_empty_rows():
    """Chunk 96 with window 1 and query block 1 (tokens 64..127) holding both
    sides of the boundary: a list with only key block 3 (tokens 192..255)
    leaves every row of block 1 without allowed keys (rows 64..95 may see
    0..95, rows 96..127 may see 96..191), so they get O = 0, LSE = -inf."""
    N, block, causal = 256, 64, (96, 1)
    g = torch.Generator().manual_seed(5)
    q, k, v = (torch.randn(1, 1, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    idx = torch.tensor([[[[0, -1], [3, -1], [1, 2], [2, 3]]]], dtype=torch.int32)
    cnt = torch.tensor([[[1, 1, 2, 2]]], dtype=torch.int32)
    o, lse = fwd_causal_check(q, k, v, idx.to(DEV), cnt.to(DEV), block, causal, "empty rows")
    assert torch.all(o[0, 0, 64:128] == 0) and torch.all(torch.isneginf(lse[0, 0, 64:128]))


def test_causal_wan13b_ar_chunks():
    """The 1.3B 480P shape generated auto-regressively in chunks of 3 latent
    frames (3 x 30 x 52 = 4680 tokens), full causal history, 90% sparsity:
    selection on all 12 heads, outputs on 2 heads."""
    wl = W.WORKLOADS["wan13b_480p"]
    q, k, v = W.make_inputs(wl, heads=[0, 7])
    causal = (3 * 30 * 52, 0)
    idx, cnt = select_causal_check(q, k, wl.block, wl.keep_bp, causal, "wan13b AR")
    fwd_causal_check(q, k, v, idx, cnt, wl.block, causal, "wan13b AR fwd")


def test_causal_fp8_forward():
    wl = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(wl)
    causal = (1024, 2)
    block = wl.block
    idx, cnt = select_causal_check(q, k, block, wl.keep_bp, causal, "tiny fp8")
    qd, kd, vd = (t.to(DEV) for t in (q, k, v))
    q8, sq = sa.sparse_attn_quant_fp8(qd, block=block)
    k8, sk = sa.sparse_attn_quant_fp8_tiles(kd, sa.SA_FP8_K, block=block)
    v8, sv = sa.sparse_attn_quant_fp8_tiles(vd, sa.SA_FP8_V, block=block)
    o, lse = sa.sparse_attn_fwd_fp8(q8, sq, k8, sk, v8, sv, idx, cnt, block=block, causal=causal)
    torch.cuda.synchronize()
    o, lse = o.cpu(), lse.cpu()
    idx_c, cnt_c = idx.cpu().numpy(), cnt.cpu().numpy()
    for h in range(q.shape[1]):
        deq = [O.dequantize_fp8_blocks(*O.quantize_fp8_blocks(widen(t[0, h]), block), block)
               for t in (q, k, v)]
        ro, rl = O.sparse_attention_causal(*deq, idx_c[0, h], cnt_c[0, h], block, TAU, *causal)
        check_out(o[0, h], None, ro, rl, rel=FP8_REL_L2, mabs=None, what=f"fp8 causal h{h}")
        assert np.array_equal(np.isneginf(lse[0, h].numpy()), np.isneginf(rl))


def test_causal_full_chunk_equals_unrestricted():
    """A single chunk covering the sequence is no restriction: the lists and
    the output equal the unrestricted calls bit for bit."""
    wl = W.WORKLOADS["tiny"]
    q, k, v = (t.to(DEV) for t in W.make_inputs(wl))
    kk = O.keep_count(wl.keep_bp, O.block_count(wl.seqlen, wl.block))
    i0, c0 = sa.sparse_attn_select(q, k, kk)
    i1, c1 = sa.sparse_attn_select(q, k, kk, causal=(wl.seqlen, 0))
    o0, l0 = sa.sparse_attn_fwd(q, k, v, i0, c0)
    o1, l1 = sa.sparse_attn_fwd(q, k, v, i1, c1, causal=(wl.seqlen, 0))
    torch.cuda.synchronize()
    assert torch.equal(i0, i1) and torch.equal(c0, c1)
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16)) and torch.equal(l0, l1)


@pytest.mark.parametrize("N,causal", [(1064, (300, 1)), (4160, (1000, 0)), (8200, (2000, 2))])
def test_causal_block128_tail_sub_tile_past_end(N, causal):
    """Block 128 with N mod 128 in (0, 64] under a window: the last block's
    second 64-token sub-tile lies past N, and chunk boundaries fall inside
    blocks."""
    g = torch.Generator().manual_seed(N + 17)
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    idx, cnt = select_causal_check(q, k, 128, 3000, causal, f"b128 tail N={N} {causal}")
    fwd_causal_check(q, k, v, idx, cnt, 128, causal, f"b128 tail fwd N={N} {causal}")

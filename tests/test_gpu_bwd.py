"""GPU parity of the sparse-branch backward through the C ABI against the
fp64 oracle on identical seeded inputs.

The GPU takes the forward's own bf16 O and fp32 LSE, rounds P and dS to bf16
for the second products and rounds dQ, dK, dV to bf16, each a relative
error of at most 2^-9 per term; these average out in the sums, and the
measured rel-L2 is a few 1e-3.  Bars per gradient and head: rel-L2 <= 1e-2
(the forward's bf16 bar) and max |err| <= 2e-2 max |ref| (the forward's
max-abs bar relative to the gradient's scale, which the inputs do not fix).
Under a causal window the forward and backward take the window from the
descriptor and the oracle is its causal backward."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_23153_amd as sa
import workloads as W
from gpu_helpers import rel_l2, say, widen

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


def run_bwd(q, k, v, idx, cnt, block, seed, causal=None):
    g = torch.Generator().manual_seed(seed)
    do = torch.randn(q.shape, generator=g).to(torch.bfloat16)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    idxd, cntd = idx.to(DEV), cnt.to(DEV)
    o, lse = sa.sparse_attn_fwd(qd, kd, vd, idxd, cntd, block=block, causal=causal)
    dq, dk, dv = sa.sparse_attn_bwd(qd, kd, vd, o, dod, lse, idxd, cntd, block=block,
                                    causal=causal)
    torch.cuda.synchronize()
    return do, dq.cpu(), dk.cpu(), dv.cpu()


def check_grads(q, k, v, do, idx, cnt, block, dq, dk, dv, what, heads=None, causal=None):
    B, H = q.shape[:2]
    idx_c, cnt_c = idx.numpy(), cnt.numpy()
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            args = (widen(q[b, h]), widen(k[b, h]), widen(v[b, h]), widen(do[b, h]),
                    idx_c[b, h], cnt_c[b, h], block, TAU)
            ref = (O.sparse_attention_backward(*args) if causal is None else
                   O.sparse_attention_backward_causal(*args, *causal))
            msg = []
            for name, got, r in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
                gg = got[b, h].to(torch.float64).numpy()
                e = rel_l2(gg, r)
                scale = float(np.abs(r).max()) or 1.0
                m = float(np.abs(gg - r).max()) / scale
                msg.append(f"{name} rel_l2={e:.2e} max/scale={m:.2e}")
                assert e <= 1e-2 and m <= 2e-2, (what, b, h, name, e, m)
                # exact zeros where the oracle has no contribution
                zero = np.all(r == 0, axis=1)
                assert np.all(gg[zero] == 0), (what, name, "nonzero where nothing contributes")
            say(f"  {what} b{b} h{h}: " + "  ".join(msg))


def test_bwd_tiny():
    wl = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(wl)
    nb = O.block_count(wl.seqlen, wl.block)
    kk = O.keep_count(wl.keep_bp, nb)
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), kk, block=wl.block)
    idx, cnt = idx.cpu(), cnt.cpu()
    do, dq, dk, dv = run_bwd(q, k, v, idx, cnt, wl.block, 1)
    check_grads(q, k, v, do, idx, cnt, wl.block, dq, dk, dv, "tiny")


@pytest.mark.parametrize("N,block", [(1000, 64), (1000, 128), (200, 64), (4096, 128)])
def test_bwd_ragged_lists_with_empty_rows(N, block):
    """Random ragged lists (about 15% empty), ragged last block: dQ = 0 for
    empty lists, dK = dV = 0 for keys nobody selected."""
    g = torch.Generator().manual_seed(N * 3 + block)
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    nb = O.block_count(N, block)
    kmax = min(nb, 7)
    idx = np.full((1, 2, nb, kmax), -1, dtype=np.int32)
    cnt = np.zeros((1, 2, nb), dtype=np.int32)
    for h in range(2):
        ii, cc = W.random_block_lists(nb, nb, kmax, seed=N + block + h, p_empty=0.15)
        idx[0, h], cnt[0, h] = ii, cc
    idx, cnt = torch.from_numpy(idx), torch.from_numpy(cnt)
    do, dq, dk, dv = run_bwd(q, k, v, idx, cnt, block, 2)
    check_grads(q, k, v, do, idx, cnt, block, dq, dk, dv, f"ragged N={N} b={block}")


def test_bwd_deterministic():
    wl = W.WORKLOADS["tiny"]
    q, k, v = (t.to(DEV) for t in W.make_inputs(wl))
    kk = O.keep_count(wl.keep_bp, O.block_count(wl.seqlen, wl.block))
    idx, cnt = sa.sparse_attn_select(q, k, kk)
    o, lse = sa.sparse_attn_fwd(q, k, v, idx, cnt)
    do = torch.randn_like(q)
    a = sa.sparse_attn_bwd(q, k, v, o, do, lse, idx, cnt)
    b = sa.sparse_attn_bwd(q, k, v, o, do, lse, idx, cnt)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))


def test_bwd_full_size_one_head():
    """The 14B-720P layer (40 heads, 75,600 tokens, 36 of 1182 blocks): the
    whole backward runs in one launch; head 0 is checked against the oracle
    (all its query blocks, since dK and dV gather from every one), every
    gradient checked finite."""
    wl = W.WORKLOADS["wan14b_720p"]
    q, k, v = W.make_inputs(wl)
    kk = O.keep_count(wl.keep_bp, O.block_count(wl.seqlen, wl.block))
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), kk, block=wl.block)
    idx, cnt = idx.cpu(), cnt.cpu()
    do, dq, dk, dv = run_bwd(q, k, v, idx, cnt, wl.block, 3)
    for t in (dq, dk, dv):
        assert torch.isfinite(t.float()).all()
    check_grads(q, k, v, do, idx, cnt, wl.block, dq, dk, dv, "14B-720P", heads=[0])


# ---- causal window ----------------------------------------------------------
@pytest.mark.parametrize("causal", [(1024, 0), (1024, 2), (2048, 1)])
def test_bwd_causal_tiny(causal):
    """4 frames of 32 x 32 tokens in chunks of 1 or 2 frames, the lists from
    the causal selection."""
    wl = W.WORKLOADS["tiny"]
    q, k, v = W.make_inputs(wl)
    kk = O.keep_count(wl.keep_bp, O.block_count(wl.seqlen, wl.block))
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), kk, block=wl.block, causal=causal)
    idx, cnt = idx.cpu(), cnt.cpu()
    do, dq, dk, dv = run_bwd(q, k, v, idx, cnt, wl.block, 4, causal=causal)
    check_grads(q, k, v, do, idx, cnt, wl.block, dq, dk, dv, f"causal tiny {causal}",
                causal=causal)


@pytest.mark.parametrize("N,block,causal", [(1000, 64, (600, 1)), (1000, 128, (300, 0)),
                                            (777, 64, (777, 0)), (3000, 64, (1000, 2))])
def test_bwd_causal_unaligned_chunks(N, block, causal):
    """Chunk boundaries inside blocks and a ragged last block, causal lists."""
    g = torch.Generator().manual_seed(N + block + causal[0])
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    kk = O.keep_count(1500, O.block_count(N, block))
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), kk, block=block, causal=causal)
    idx, cnt = idx.cpu(), cnt.cpu()
    do, dq, dk, dv = run_bwd(q, k, v, idx, cnt, block, 5, causal=causal)
    check_grads(q, k, v, do, idx, cnt, block, dq, dk, dv, f"causal N={N} b={block} {causal}",
                causal=causal)


def test_bwd_causal_rows_without_allowed_keys():
    """Chunk 96, window 1: query block 1 listing only key block 3 leaves all
    its rows without allowed keys (LSE = -inf): dQ = 0 there and nothing
    reaches dK, dV of block 3 from them."""
    N, block, causal = 256, 64, (96, 1)
    g = torch.Generator().manual_seed(6)
    q, k, v = (torch.randn(1, 1, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    idx = torch.tensor([[[[0, -1], [3, -1], [1, 2], [2, 3]]]], dtype=torch.int32)
    cnt = torch.tensor([[[1, 1, 2, 2]]], dtype=torch.int32)
    do, dq, dk, dv = run_bwd(q, k, v, idx, cnt, block, 7, causal=causal)
    assert torch.all(dq[0, 0, 64:128] == 0)
    check_grads(q, k, v, do, idx, cnt, block, dq, dk, dv, "causal empty rows", causal=causal)


def test_bwd_causal_full_chunk_equals_unrestricted():
    """One chunk covering the sequence is no restriction: the gradients equal
    the unrestricted call bit for bit."""
    wl = W.WORKLOADS["tiny"]
    q, k, v = (t.to(DEV) for t in W.make_inputs(wl))
    kk = O.keep_count(wl.keep_bp, O.block_count(wl.seqlen, wl.block))
    idx, cnt = sa.sparse_attn_select(q, k, kk)
    o, lse = sa.sparse_attn_fwd(q, k, v, idx, cnt)
    do = torch.randn_like(q)
    a = sa.sparse_attn_bwd(q, k, v, o, do, lse, idx, cnt)
    b = sa.sparse_attn_bwd(q, k, v, o, do, lse, idx, cnt, causal=(wl.seqlen, 0))
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int16), y.view(torch.int16))


@pytest.mark.parametrize("N", [1064, 4160])
def test_bwd_block128_tail_sub_tile_past_end(N):
    """Block 128 with N mod 128 in (0, 64]: the last block's second 64-row
    sub-tile lies past N for the dQ query tiles and the dK/dV key tiles;
    lists often include the tail block."""
    from test_gpu_parity import tail_lists
    g = torch.Generator().manual_seed(N + 9)
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    nb = O.block_count(N, 128)
    idx, cnt = tail_lists(nb, min(nb, 7), seed=N + 4)
    do, dq, dk, dv = run_bwd(q, k, v, idx, cnt, 128, 8)
    check_grads(q, k, v, do, idx, cnt, 128, dq, dk, dv, f"b128 tail N={N}")


@pytest.mark.parametrize("N,block,causal", [(1064, 128, (300, 1)), (4160, 128, (1000, 0))])
def test_bwd_block128_tail_causal(N, block, causal):
    from test_gpu_parity import tail_lists
    g = torch.Generator().manual_seed(N + 11)
    q, k, v = (torch.randn(1, 2, N, 128, generator=g).to(torch.bfloat16) for _ in range(3))
    kk = O.keep_count(3000, O.block_count(N, block))
    idx, cnt = sa.sparse_attn_select(q.to(DEV), k.to(DEV), kk, block=block, causal=causal)
    idx, cnt = idx.cpu(), cnt.cpu()
    do, dq, dk, dv = run_bwd(q, k, v, idx, cnt, block, 9, causal=causal)
    check_grads(q, k, v, do, idx, cnt, block, dq, dk, dv, f"b128 tail causal N={N} {causal}",
                causal=causal)


def test_bwd_strided_token_major_layout():
    """[B, N, H, d] storage viewed as [B, H, N, d] for every input and
    gradient (strides (N*H*d, d, H*d))."""
    from test_gpu_parity import tail_lists
    g = torch.Generator().manual_seed(13)
    N, H = 1500, 3
    base = [torch.randn(1, N, H, 128, generator=g).to(torch.bfloat16) for _ in range(4)]
    q, k, v, do = (t.permute(0, 2, 1, 3) for t in base)
    nb = O.block_count(N, 64)
    idx, cnt = tail_lists(nb, 6, seed=14, H=H)
    qd, kd, vd, dod = (t.to(DEV).permute(0, 2, 1, 3) for t in base)
    idxd, cntd = idx.to(DEV), cnt.to(DEV)
    o = torch.empty(1, N, H, 128, dtype=torch.bfloat16, device=DEV).permute(0, 2, 1, 3)
    o, lse = sa.sparse_attn_fwd(qd, kd, vd, idxd, cntd, o=o)
    grads = [torch.empty(1, N, H, 128, dtype=torch.bfloat16, device=DEV).permute(0, 2, 1, 3)
             for _ in range(3)]
    dq, dk, dv = sa.sparse_attn_bwd(qd, kd, vd, o, dod, lse, idxd, cntd, dq=grads[0],
                                    dk=grads[1], dv=grads[2])
    torch.cuda.synchronize()
    assert dq.stride() == qd.stride()
    check_grads(q, k, v, do, idx, cnt, 64, dq.cpu(), dk.cpu(), dv.cpu(), "strided [B,N,H,d]")

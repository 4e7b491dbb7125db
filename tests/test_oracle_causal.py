"""Pins of the oracle's causal-window restriction (paper §1, extension to
auto-regressive video diffusion) against facts independent of it: brute-force
enumeration of the allowed token pairs and candidate blocks, the reduction to
the unrestricted selection for one chunk, dense masked attention from a
library routine when every candidate is kept, the block-diagonal special
case, and a hand-built empty row."""
import math

import numpy as np
import pytest
import torch

import oracle as O


def brute_allowed(n, chunk, window):
    ok = np.zeros((n, n), bool)
    for t in range(n):
        for u in range(n):
            ct, cu = t // chunk, u // chunk
            ok[t, u] = cu <= ct and (window == 0 or cu >= ct - window + 1)
    return ok


@pytest.mark.parametrize("n,chunk,window", [(37, 5, 0), (37, 5, 2), (40, 8, 1), (23, 30, 0),
                                            (50, 7, 3)])
def test_allowed_and_candidate_ranges_by_enumeration(n, chunk, window):
    ok = brute_allowed(n, chunk, window)
    lo, hi = O.allowed_range(n, chunk, window)
    for t in range(n):
        assert np.array_equal(np.nonzero(ok[t])[0], np.arange(lo[t], hi[t]))
    block = 6
    nb = -(-n // block)
    jlo, jhi = O.candidate_range(n, block, chunk, window)
    for i in range(nb):
        cand = [j for j in range(nb)
                if ok[i * block:min(n, (i + 1) * block), j * block:min(n, (j + 1) * block)].any()]
        assert cand == list(range(jlo[i], jhi[i])), (i, cand)


def test_one_chunk_is_the_unrestricted_selection_and_attention():
    rng = np.random.default_rng(1)
    n, d, block = 300, 16, 32
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    idx, cnt = O.select_causal(q, k, block, 3000, chunk=n, window=0)
    ref_idx, ref_cnt = O.select_head(q, k, block, 3000)
    assert np.array_equal(idx, ref_idx) and np.array_equal(cnt, ref_cnt)
    o, lse = O.sparse_attention_causal(q, k, v, idx, cnt, block, 0.25, chunk=n, window=0)
    ro, rl = O.sparse_attention(q, k, v, ref_idx, ref_cnt, block, 0.25)
    assert np.allclose(o, ro, rtol=1e-13, atol=1e-13) and np.allclose(lse, rl, rtol=1e-13)


@pytest.mark.parametrize("chunk,window", [(50, 0), (50, 2), (37, 1)])
def test_all_candidates_kept_equals_dense_masked_attention(chunk, window):
    rng = np.random.default_rng(2)
    n, d, block, tau = 230, 8, 16, 0.3
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    idx, cnt = O.select_causal(q, k, block, 10000, chunk, window)
    jlo, jhi = O.candidate_range(n, block, chunk, window)
    assert np.array_equal(cnt, jhi - jlo)
    o, lse = O.sparse_attention_causal(q, k, v, idx, cnt, block, tau, chunk, window)
    mask = torch.from_numpy(brute_allowed(n, chunk, window))
    tq, tk, tv = (torch.from_numpy(x)[None, None] for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=mask[None, None],
                                                           scale=tau)[0, 0].numpy()
    logits = (tau * (torch.from_numpy(q) @ torch.from_numpy(k).T)).masked_fill(~mask, -math.inf)
    assert np.allclose(o, ref, rtol=1e-12, atol=1e-12)
    assert np.allclose(lse, torch.logsumexp(logits, dim=1).numpy(), rtol=1e-12, atol=1e-12)


def test_window_one_chunk_equal_block_is_block_diagonal():
    rng = np.random.default_rng(3)
    n, d, block, tau = 160, 8, 32, 0.5
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    idx, cnt = O.select_causal(q, k, block, 5000, chunk=block, window=1)
    assert np.array_equal(cnt, np.ones(5)) and np.array_equal(idx[:, 0], np.arange(5))
    assert (idx[:, 1:] == -1).all()
    o, _ = O.sparse_attention_causal(q, k, v, idx, cnt, block, tau, chunk=block, window=1)
    for i in range(5):
        r = slice(i * block, (i + 1) * block)
        z = tau * q[r] @ k[r].T
        p = np.exp(z - z.max(1, keepdims=True))
        assert np.allclose(o[r], (p / p.sum(1, keepdims=True)) @ v[r], rtol=1e-13, atol=1e-13)


def test_rows_without_allowed_selected_keys_are_empty():
    """Chunk boundary in the middle of query block 1 (chunk 24, block 16,
    window 1): rows 16..23 may attend keys 0..23 only, rows 24..31 keys
    24..47 only.  A list holding just key block 2 (keys 32..47) leaves rows
    16..23 with nothing: O = 0, LSE = -inf there, finite elsewhere."""
    rng = np.random.default_rng(4)
    n, d, block = 48, 4, 16
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    idx = np.array([[0], [2], [2]], dtype=np.int32)
    cnt = np.array([1, 1, 1], dtype=np.int32)
    o, lse = O.sparse_attention_causal(q, k, v, idx, cnt, block, 1.0, chunk=24, window=1)
    assert np.all(o[16:24] == 0) and np.all(lse[16:24] == -np.inf)
    assert np.all(np.isfinite(lse[24:32])) and np.all(np.isfinite(lse[:16]))
    # rows 24..31 see keys 32..47 (their chunk is 24..47, and block 2 is inside it)
    z = q[24:32] @ k[32:48].T
    p = np.exp(z - z.max(1, keepdims=True))
    assert np.allclose(o[24:32], (p / p.sum(1, keepdims=True)) @ v[32:48], rtol=1e-13)

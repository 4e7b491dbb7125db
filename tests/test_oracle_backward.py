"""Pins of the oracle's backward pass against facts independent of it: torch
autograd through a dense attention whose scores outside the selected blocks
are masked (fp64), central finite differences of a scalar loss on a tiny
case, the all-blocks case against autograd through torch's SDPA, and the
zero contribution of empty lists.  The causal-window backward is pinned the
same way with the window's token mask added, including a row left without
allowed keys, and reduces to the unrestricted backward for one chunk."""
import numpy as np
import pytest
import torch

import oracle as O


def masked_autograd(q, k, v, do, idx, cnt, block, tau, token_mask=None):
    n = q.shape[0]
    allowed = np.zeros((n, n), bool)
    for i in range(O.block_count(n, block)):
        r = slice(i * block, min((i + 1) * block, n))
        for j in idx[i, :cnt[i]]:
            allowed[r, j * block:min((j + 1) * block, n)] = True
    if token_mask is not None:
        allowed &= token_mask
    tq, tk, tv = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v))
    z = tau * tq @ tk.T
    z = z.masked_fill(~torch.from_numpy(allowed), -float("inf"))
    p = torch.softmax(z, dim=1)
    p = torch.nan_to_num(p, nan=0.0)            # fully masked rows (empty lists)
    o = p @ tv
    o.backward(torch.tensor(do, dtype=torch.float64))
    return tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


@pytest.mark.parametrize("n,block,kk", [(96, 16, 2), (100, 16, 3), (64, 32, 1)])
def test_matches_autograd_of_the_masked_dense_attention(n, block, kk):
    rng = np.random.default_rng(n + block)
    d, tau = 8, 0.4
    q, k, v, do = (rng.standard_normal((n, d)) for _ in range(4))
    nb = O.block_count(n, block)
    idx = np.full((nb, kk), -1, np.int32)
    cnt = np.full(nb, kk, np.int32)
    for i in range(nb):
        idx[i] = np.sort(rng.choice(nb, kk, replace=False))
    cnt[1] = 0                                   # an empty list
    idx[1] = -1
    got = O.sparse_attention_backward(q, k, v, do, idx, cnt, block, tau)
    ref = masked_autograd(q, k, v, do, idx, cnt, block, tau)
    for g, r in zip(got, ref):
        assert np.allclose(g, r, rtol=1e-12, atol=1e-12)
    assert np.all(got[0][block:2 * block] == 0)   # rows of the empty list


def test_finite_differences():
    rng = np.random.default_rng(7)
    n, d, block, tau = 20, 3, 8, 0.7
    q, k, v, do = (rng.standard_normal((n, d)) for _ in range(4))
    idx = np.array([[0, 2], [1, -1], [0, 1]], np.int32)
    cnt = np.array([2, 1, 2], np.int32)
    dq, dk, dv = O.sparse_attention_backward(q, k, v, do, idx, cnt, block, tau)

    def loss(q_, k_, v_):
        o, _ = O.sparse_attention(q_, k_, v_, idx, cnt, block, tau)
        return float(np.sum(o * do))

    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for (a, b) in [(0, 0), (5, 2), (17, 1), (9, 0)]:
            xp, xm = x.copy(), x.copy()
            xp[a, b] += h
            xm[a, b] -= h
            args_p = [q, k, v]
            args_m = [q, k, v]
            pos = "qkv".index(name)
            args_p[pos], args_m[pos] = xp, xm
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            assert abs(fd - g[a, b]) < 1e-7 * max(1.0, abs(fd)), (name, a, b, fd, g[a, b])


def test_all_blocks_equals_sdpa_autograd():
    rng = np.random.default_rng(9)
    n, d, block, tau = 70, 8, 16, 0.3
    q, k, v, do = (rng.standard_normal((n, d)) for _ in range(4))
    nb = O.block_count(n, block)
    idx = np.tile(np.arange(nb, dtype=np.int32), (nb, 1))
    cnt = np.full(nb, nb, np.int32)
    got = O.sparse_attention_backward(q, k, v, do, idx, cnt, block, tau)
    tq, tk, tv = (torch.tensor(x, requires_grad=True) for x in (q, k, v))
    o = torch.nn.functional.scaled_dot_product_attention(tq[None], tk[None], tv[None],
                                                         scale=tau)[0]
    o.backward(torch.from_numpy(do))
    for g, r in zip(got, (tq.grad, tk.grad, tv.grad)):
        assert np.allclose(g, r.numpy(), rtol=1e-12, atol=1e-12)


def causal_token_mask(n, chunk, window):
    """Brute force over token pairs: key u allowed for query t iff its chunk
    lies in the last `window` chunks up to t's own (every earlier one if 0)."""
    m = np.zeros((n, n), bool)
    for t in range(n):
        for u in range(n):
            ct, cu = t // chunk, u // chunk
            m[t, u] = cu <= ct and (window == 0 or cu > ct - window)
    return m


@pytest.mark.parametrize("n,block,chunk,window", [(96, 16, 24, 0), (100, 16, 30, 1),
                                                  (64, 32, 20, 2)])
def test_causal_matches_autograd_of_the_masked_dense_attention(n, block, chunk, window):
    rng = np.random.default_rng(n + chunk)
    d, tau = 8, 0.4
    q, k, v, do = (rng.standard_normal((n, d)) for _ in range(4))
    nb = O.block_count(n, block)
    kk = min(3, nb)
    idx = np.full((nb, kk), -1, np.int32)
    cnt = np.full(nb, kk, np.int32)
    for i in range(nb):
        idx[i] = np.sort(rng.choice(nb, kk, replace=False))
    cnt[1] = 0
    idx[1] = -1
    got = O.sparse_attention_backward_causal(q, k, v, do, idx, cnt, block, tau, chunk, window)
    ref = masked_autograd(q, k, v, do, idx, cnt, block, tau,
                          token_mask=causal_token_mask(n, chunk, window))
    for g, r in zip(got, ref):
        assert np.allclose(g, r, rtol=1e-12, atol=1e-12)


def test_causal_row_without_allowed_keys_contributes_nothing():
    """Chunk 8, window 1, block 16: query block 1 (tokens 16..31) listing only
    key block 0 leaves tokens 16..31 without allowed keys; their dQ is 0 and
    they add nothing to dK, dV (checked against the same case without them)."""
    rng = np.random.default_rng(3)
    n, d, block, tau = 32, 4, 16, 0.5
    q, k, v, do = (rng.standard_normal((n, d)) for _ in range(4))
    idx = np.array([[0], [0]], np.int32)
    cnt = np.array([1, 1], np.int32)
    dq, dk, dv = O.sparse_attention_backward_causal(q, k, v, do, idx, cnt, block, tau, 8, 1)
    assert np.all(dq[16:] == 0)
    dq0, dk0, dv0 = O.sparse_attention_backward_causal(q, k, v, do, idx,
                                                       np.array([1, 0], np.int32), block, tau,
                                                       8, 1)
    assert np.array_equal(dk, dk0) and np.array_equal(dv, dv0)
    ref = masked_autograd(q, k, v, do, idx, cnt, block, tau,
                          token_mask=causal_token_mask(n, 8, 1))
    for g, r in zip((dq, dk, dv), ref):
        assert np.allclose(g, r, rtol=1e-12, atol=1e-12)


def test_causal_one_chunk_is_the_unrestricted_backward():
    rng = np.random.default_rng(5)
    n, d, block, tau = 70, 8, 16, 0.3
    q, k, v, do = (rng.standard_normal((n, d)) for _ in range(4))
    nb = O.block_count(n, block)
    idx = np.tile(np.array([0, 2, 4], np.int32), (nb, 1))
    cnt = np.full(nb, 3, np.int32)
    a = O.sparse_attention_backward_causal(q, k, v, do, idx, cnt, block, tau, n, 0)
    b = O.sparse_attention_backward(q, k, v, do, idx, cnt, block, tau)
    for x, y in zip(a, b):
        assert np.allclose(x, y, rtol=1e-13, atol=1e-13)


def test_causal_finite_differences():
    rng = np.random.default_rng(11)
    n, d, block, tau, chunk, window = 24, 3, 8, 0.7, 6, 2
    q, k, v, do = (rng.standard_normal((n, d)) for _ in range(4))
    idx = np.array([[0, 1], [0, 2], [1, 2]], np.int32)
    cnt = np.array([2, 2, 2], np.int32)
    dq, dk, dv = O.sparse_attention_backward_causal(q, k, v, do, idx, cnt, block, tau, chunk,
                                                    window)

    def loss(q_, k_, v_):
        o, _ = O.sparse_attention_causal(q_, k_, v_, idx, cnt, block, tau, chunk, window)
        return float(np.sum(o * do))

    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        for (a, b) in [(0, 0), (7, 2), (13, 1), (22, 0)]:
            xp, xm = x.copy(), x.copy()
            xp[a, b] += h
            xm[a, b] -= h
            args_p, args_m = [q, k, v], [q, k, v]
            pos = "qkv".index(name)
            args_p[pos], args_m[pos] = xp, xm
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            assert abs(fd - g[a, b]) < 1e-7 * max(1.0, abs(fd)), (name, a, b, fd, g[a, b])

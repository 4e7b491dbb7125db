"""Backward pass of the block-sparse attention (the sparse branch), written out
in fp64 from the chain rule (test infrastructure only; the product path never
imports this package).

The forward (paper §2 Eq. comp-sparse, §3: exact softmax attention over the
key blocks each query block selected) is, per query block i with key set U_i
(the union of its selected blocks' tokens),
    Z = tau Q_i K_U^T,  P = softmax_rows(Z),  O_i = P V_U.
Its gradients for an upstream dO (the training that needs them: §2 "Training
sparse attention" and the Stage-1 warm-up of §4.4):
    dV_U += P^T dO_i
    dP    = dO_i V_U^T
    dZ    = P o (dP - D 1^T),  D = rowsum(dO_i o O_i) = rowsum(P o dP)
    dQ_i  = tau dZ K_U,   dK_U += tau dZ^T Q_i
A query block with an empty list contributes nothing (its O is 0 and its
gradients are 0).  The selection is a discrete choice and gets no gradient.

Under a causal window (§1, auto-regressive extension; the chunk and window
readings of causal_window.py) the same chain rule runs over the allowed keys
of each row's selected blocks: P is 0 outside them, and a row without any
allowed key (O = 0, LSE = -inf) contributes nothing.
"""
from __future__ import annotations

import numpy as np

from .causal_window import allowed_range
from .sparse_attention import block_count

__all__ = ["sparse_attention_backward", "sparse_attention_backward_causal"]


def sparse_attention_backward(q, k, v, do, idx, cnt, block: int, tau: float):
    """(dQ, dK, dV) of one head, fp64, for the lists idx/cnt."""
    q, k, v, do = (np.asarray(x, np.float64) for x in (q, k, v, do))
    n = q.shape[0]
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for i in range(block_count(n, block)):
        blocks = [int(j) for j in idx[i, :int(cnt[i])]]
        if not blocks:
            continue
        rows = np.arange(i * block, min((i + 1) * block, n))
        keys = np.concatenate([np.arange(j * block, min((j + 1) * block, n)) for j in blocks])
        z = tau * (q[rows] @ k[keys].T)
        p = np.exp(z - z.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        o = p @ v[keys]
        dv[keys] += p.T @ do[rows]
        dp = do[rows] @ v[keys].T
        d = np.sum(do[rows] * o, axis=1, keepdims=True)
        dz = p * (dp - d)
        dq[rows] = tau * (dz @ k[keys])
        dk[keys] += tau * (dz.T @ q[rows])
    return dq, dk, dv


def sparse_attention_backward_causal(q, k, v, do, idx, cnt, block: int, tau: float,
                                     chunk: int, window: int):
    """(dQ, dK, dV) of one head, fp64, for the lists idx/cnt under the causal
    window (chunk tokens, window in chunks, 0 = every earlier chunk)."""
    q, k, v, do = (np.asarray(x, np.float64) for x in (q, k, v, do))
    n = q.shape[0]
    lo, hi = allowed_range(n, chunk, window)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    for i in range(block_count(n, block)):
        blocks = [int(j) for j in idx[i, :int(cnt[i])]]
        if not blocks:
            continue
        rows = np.arange(i * block, min((i + 1) * block, n))
        keys = np.concatenate([np.arange(j * block, min((j + 1) * block, n)) for j in blocks])
        allowed = (keys[None, :] >= lo[rows, None]) & (keys[None, :] < hi[rows, None])
        z = np.where(allowed, tau * (q[rows] @ k[keys].T), -np.inf)
        m = z.max(axis=1, keepdims=True)
        m = np.where(np.isfinite(m), m, 0.0)          # rows without allowed keys
        e = np.where(allowed, np.exp(z - m), 0.0)
        ssum = e.sum(axis=1, keepdims=True)
        p = e / np.where(ssum > 0, ssum, 1.0)
        o = p @ v[keys]
        dv[keys] += p.T @ do[rows]
        dp = do[rows] @ v[keys].T
        d = np.sum(do[rows] * o, axis=1, keepdims=True)
        dz = p * (dp - d)
        dq[rows] = tau * (dz @ k[keys])
        dk[keys] += tau * (dz.T @ q[rows])
    return dq, dk, dv

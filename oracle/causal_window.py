"""Causal-window (auto-regressive) restriction of block-sparse attention,
written out from its definition in fp64 (test infrastructure only; the
product path never imports this package).

Paper §1 (extension to auto-regressive video diffusion): the compensated
sparse attention can be restricted to a causal window.  Readings where the
paper is silent (stated in the design notes):
  * Tokens are grouped into chunks of C consecutive tokens (the latent frames
    generated together, C = frames per chunk x tokens per frame).  Query t,
    in chunk c(t) = t // C, may attend key u iff c(u) lies in
    [c(t) - W + 1, c(t)]; W is the window in chunks, W = 0 meaning every
    earlier chunk.  The allowed keys of t form one token range
    [lo(t), hi(t)).
  * The candidate key blocks of query block i are those holding an allowed
    key of some query of the block.  lo and hi never decrease with t, so the
    candidates form the block range [lo(first) // b, ceil(hi(last) / b)).
  * Selection: top-k of the pooled block scores over the candidates only,
    k_i = min(k, number of candidates), ties to the lower index, lists
    ascending and padded with -1 to k.
  * Attention: exact softmax over the allowed keys of the selected blocks;
    a row with none of them gets O = 0 and LSE = -inf.
"""
from __future__ import annotations

import numpy as np

from .sparse_attention import (NEG_INF, block_count, block_scores, keep_count,
                               topk_ascending)

__all__ = ["allowed_range", "candidate_range", "select_causal", "sparse_attention_causal"]


def allowed_range(n: int, chunk: int, window: int):
    """(lo, hi) int64 [n]: the allowed key tokens [lo(t), hi(t)) of every query."""
    if chunk < 1 or window < 0:
        raise ValueError("chunk >= 1 and window >= 0")
    t = np.arange(n, dtype=np.int64)
    c = t // chunk
    first = np.zeros(n, np.int64) if window == 0 else np.maximum(c - window + 1, 0)
    return first * chunk, np.minimum((c + 1) * chunk, n)


def candidate_range(n: int, block: int, chunk: int, window: int):
    """(jlo, jhi) int64 [nqb]: candidate key blocks [jlo, jhi) of every query block."""
    lo, hi = allowed_range(n, chunk, window)
    nqb = block_count(n, block)
    first = np.arange(nqb, dtype=np.int64) * block
    last = np.minimum(first + block, n) - 1
    return lo[first] // block, -(-hi[last] // block)


def select_causal(q, k, block: int, keep_bp: int, chunk: int, window: int):
    """Row top-k restricted to the candidates -> (idx [nqb, kk] int32 padded
    with -1, cnt [nqb] int32), kk = keep_count over all key blocks."""
    n = q.shape[0]
    s = block_scores(q, k, block)
    nqb, nkb = s.shape
    kk = keep_count(keep_bp, nkb)
    jlo, jhi = candidate_range(n, block, chunk, window)
    idx = np.full((nqb, kk), -1, dtype=np.int32)
    cnt = np.zeros(nqb, dtype=np.int32)
    for i in range(nqb):
        ki = int(min(kk, jhi[i] - jlo[i]))
        sel = topk_ascending(s[i, jlo[i]:jhi[i]], ki) + jlo[i]
        idx[i, :ki] = sel
        cnt[i] = ki
    return idx, cnt


def sparse_attention_causal(q, k, v, idx, cnt, block: int, tau: float, chunk: int,
                            window: int, qblocks=None):
    """O_t = sum_u softmax_u(tau q_t.k_u) v_u over the allowed keys u of the
    selected blocks of t's query block -> (O [n, d], LSE [n]) in fp64."""
    n = q.shape[0]
    lo, hi = allowed_range(n, chunk, window)
    out = np.zeros((n, v.shape[1]), dtype=np.float64)
    lse = np.full(n, NEG_INF, dtype=np.float64)
    for i in (range(block_count(n, block)) if qblocks is None else qblocks):
        rows = np.arange(i * block, min((i + 1) * block, n))
        blocks = idx[i, :int(cnt[i])]
        if len(blocks) == 0:
            continue
        keys = np.concatenate([np.arange(j * block, min((j + 1) * block, n)) for j in blocks])
        z = tau * (q[rows] @ k[keys].T)
        allowed = (keys[None, :] >= lo[rows, None]) & (keys[None, :] < hi[rows, None])
        z = np.where(allowed, z, NEG_INF)
        m = z.max(axis=1, keepdims=True)
        has = np.isfinite(m[:, 0])
        ms = np.where(np.isfinite(m), m, 0.0)
        e = np.where(allowed, np.exp(z - ms), 0.0)
        ssum = e.sum(axis=1, keepdims=True)
        o = np.where(has[:, None], (e / np.where(ssum > 0, ssum, 1.0)) @ v[keys], 0.0)
        out[rows] = o
        lse[rows] = np.where(has, (ms + np.log(np.where(ssum > 0, ssum, 1.0)))[:, 0], NEG_INF)
    return out, lse

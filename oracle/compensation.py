"""Compensation branch and gate epilogue of compensated sparse attention,
written out from the paper's definition in fp64 (test infrastructure only;
the product path never imports this package).

Paper §2 Eq. comp-sparse adds a gated compensation branch to the sparse
branch A_M; §4.1 defines it as a low-rank branch with a token-wise gate:

  q~_i = R_r(p_i) silu(P_q q_i^norm),   k~_j = R_r(p_j) silu(P_k k_j^norm)
  C = sum_j k~_j v_j^T                      (r x d per head)
  O_lr,i = RMSNorm(q~_i^T C)
  O_i = O_s,i + g_i * rms(O_s,i) * O_lr,i

with rank r = 64 (the paper's hyperparameter table), silu the pointwise
nonlinearity, and R_r the rotation by the first r coordinates of the
backbone's 3D RoPE schedule.  Readings where the paper is silent (stated in
the design notes):
  * R_r acts on consecutive coordinate pairs (2m, 2m+1), m < r/2, rotating
    each by its angle theta_{i,m}; the schedule is an input table of
    (cos theta, sin theta) per token and pair (fp32 values, widened here).
  * RMSNorm(y) = y / sqrt(mean(y^2) + eps) * gamma with a per-head weight
    gamma (ones when absent); rms(x) = sqrt(mean(x^2)) without epsilon.
  * The gate g_i is an input per (batch, head, token).
  * Under a causal window (§1, auto-regressive extension; chunk and window
    as in causal_window.py) the branch sees the same keys as the sparse
    branch: the state of query t sums k~_j v_j^T over the keys j of chunks
    [c(t) - W + 1, c(t)] (every earlier chunk when W = 0), so it depends only
    on t's chunk: one state per chunk.
"""
from __future__ import annotations

import numpy as np

__all__ = ["silu", "rope_rotate", "comp_features", "comp_state", "comp_lowrank",
           "comp_combine", "compensated_output", "comp_state_causal", "comp_lowrank_causal",
           "compensated_output_causal"]


def silu(x):
    """silu(x) = x * sigmoid(x), evaluated stably for either sign."""
    x = np.asarray(x, dtype=np.float64)
    e = np.exp(-np.abs(x))
    sig = np.where(x >= 0, 1.0 / (1.0 + e), e / (1.0 + e))
    return x * sig


def rope_rotate(x, rope):
    """Rotate consecutive coordinate pairs of x [N, r] by the angles whose
    (cos, sin) are rope [N, r/2, 2]: (a, b) -> (a cos - b sin, a sin + b cos)."""
    x = np.asarray(x, dtype=np.float64)
    c, s = rope[..., 0].astype(np.float64), rope[..., 1].astype(np.float64)
    a, b = x[:, 0::2], x[:, 1::2]
    out = np.empty_like(x)
    out[:, 0::2] = a * c - b * s
    out[:, 1::2] = a * s + b * c
    return out


def comp_features(x_norm, proj, rope):
    """R_r(p) silu(P x^norm) for every token: x_norm [N, d], proj [r, d],
    rope [N, r/2, 2] -> [N, r]."""
    return rope_rotate(silu(np.asarray(x_norm, np.float64) @ np.asarray(proj, np.float64).T), rope)


def comp_state(k_norm, v, pk, rope):
    """C = sum_j k~_j v_j^T  ->  [r, d]."""
    kt = comp_features(k_norm, pk, rope)
    return kt.T @ np.asarray(v, np.float64)


def comp_lowrank(q_norm, pq, rope, state, gamma=None, eps=1e-6):
    """O_lr = RMSNorm(q~^T C) for every token -> [N, d]."""
    y = comp_features(q_norm, pq, rope) @ np.asarray(state, np.float64)
    ms = np.mean(y * y, axis=1, keepdims=True)
    out = y / np.sqrt(ms + eps)
    if gamma is not None:
        out = out * np.asarray(gamma, np.float64)[None, :]
    return out


def comp_combine(o_s, o_lr, gate):
    """O = O_s + g * rms(O_s) * O_lr, rms over the head dimension."""
    o_s = np.asarray(o_s, np.float64)
    r = np.sqrt(np.mean(o_s * o_s, axis=1, keepdims=True))
    return o_s + np.asarray(gate, np.float64)[:, None] * r * o_lr


def compensated_output(o_s, q_norm, k_norm, v, pq, pk, rope, gate, gamma=None, eps=1e-6):
    """The full gated compensation of one head."""
    state = comp_state(k_norm, v, pk, rope)
    return comp_combine(o_s, comp_lowrank(q_norm, pq, rope, state, gamma, eps), gate)


def comp_state_causal(k_norm, v, pk, rope, chunk: int, window: int):
    """One state per query chunk c: the sum of k~_j v_j^T over the keys of
    chunks [c - window + 1, c] (every chunk up to c if window == 0)
    -> [nc, r, d], nc = ceil(N / chunk)."""
    if chunk < 1 or window < 0:
        raise ValueError("chunk >= 1 and window >= 0")
    kt = comp_features(k_norm, pk, rope)
    v = np.asarray(v, np.float64)
    n = kt.shape[0]
    nc = -(-n // chunk)
    per = [kt[c * chunk:(c + 1) * chunk].T @ v[c * chunk:(c + 1) * chunk] for c in range(nc)]
    out = np.zeros((nc,) + per[0].shape)
    for c in range(nc):
        lo = 0 if window == 0 else max(0, c - window + 1)
        for c2 in range(lo, c + 1):
            out[c] += per[c2]
    return out


def comp_lowrank_causal(q_norm, pq, rope, states, chunk: int, gamma=None, eps=1e-6):
    """O_lr = RMSNorm(q~_t^T C_(t // chunk)) for every token -> [N, d]."""
    qt = comp_features(q_norm, pq, rope)
    y = np.empty((qt.shape[0], states.shape[2]))
    for c in range(states.shape[0]):
        y[c * chunk:(c + 1) * chunk] = qt[c * chunk:(c + 1) * chunk] @ states[c]
    ms = np.mean(y * y, axis=1, keepdims=True)
    out = y / np.sqrt(ms + eps)
    if gamma is not None:
        out = out * np.asarray(gamma, np.float64)[None, :]
    return out


def compensated_output_causal(o_s, q_norm, k_norm, v, pq, pk, rope, gate, chunk: int,
                              window: int, gamma=None, eps=1e-6):
    """The gated compensation of one head under the causal window."""
    states = comp_state_causal(k_norm, v, pk, rope, chunk, window)
    return comp_combine(o_s, comp_lowrank_causal(q_norm, pq, rope, states, chunk, gamma, eps),
                        gate)

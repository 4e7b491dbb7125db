"""Seeded synthetic inputs for block-sparse attention at video-DiT shapes.

This module only draws numbers: it holds none of the attention or selection
arithmetic, and it is shared by the GPU path's tests/bench and the CPU oracle
so that both consume identical bf16 bits.

Every (batch, head) slice is generated independently from its own seed, so a
single head can be regenerated cheaply (the oracle checks sampled heads of the
largest workloads that way).  Tokens are the latent grid (T, Hg, Wg) flattened
t-major (x fastest), as a video DiT lays out its spatiotemporal tokens.

Generators (recipes are stated in words in the design notes as well):

``normal``      Q, K, V ~ N(0, 1).
``positional``  a smooth 3D positional signal shared by Q and K of one head:
                every channel is one random sinusoid over the grid,
                P[n, c] = sqrt(2) sin(w_c . (t, y, x)_n + phi_c), with
                w_c ~ N(0, 0.25^2 I) rad per grid step and phi_c ~ U[0, 2 pi),
                so that P_t . P_u ~ sum_c cos(w_c . (p_t - p_u)) decays with 3D
                grid distance (length scale ~4 steps) like the local attention
                of a video DiT; Q = P + 0.5 N(0,1), K = P + 0.5 N(0,1)
                (independent noise), V ~ N(0, 1).
``outliers``    ``positional`` plus 5 (head, channel) pairs in Q and 5 in K
                (0.1% of the H*d = 5120 pairs of a 40-head layer, rounded)
                multiplied by 20 on every token.
``locality``    random Fourier features of a Gaussian kernel over 3D grid
                distance (length scale 3 grid steps) so that logits decay with
                distance, P[n, c] = g sqrt(2/d) cos(w_c . p_n + b_c), w_c ~
                N(0, I / 3^2), b_c ~ U[0, 2 pi), g^2 = 8 / tau (peak logit
                about 8); Q = P + 0.5 N, K = P + 0.5 N; plus long-range hot
                blocks: 2% of the key blocks and 2% of the query blocks (64
                tokens) each get g * u_c added, u_c one of 8 random orthonormal
                directions; V ~ N(0, 1).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

__all__ = ["Workload", "WORKLOADS", "make_head", "make_inputs", "random_block_lists",
           "softmax_scale", "rope_pairs_wan", "rope_table", "comp_params",
           "LINEAR_SHAPES", "linear_inputs"]


def softmax_scale(d: int) -> float:
    """fp32 value of 1/sqrt(d), as the caller passes it to the kernels."""
    return float(np.float32(1.0 / math.sqrt(d)))


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads: int
    grid: tuple            # (T, Hg, Wg) latent grid
    head_dim: int
    block: int
    keep_bp: int           # keep ratio in basis points (1000 = 10%)
    gen: str
    seed: int
    sweep: tuple = field(default=())   # ((block, keep_bp), ...) for sweeps

    @property
    def seqlen(self) -> int:
        t, h, w = self.grid
        return t * h * w


WORKLOADS = {
    # B1 H2 N4096 (4x32x32), N(0,1), block 64, keep 10% -> top-7 of 64
    "tiny": Workload("tiny", 1, 2, (4, 32, 32), 128, 64, 1000, "normal", 0),
    # Wan2.1-T2V-1.3B 480P layer: H12 N32760 (21x30x52), 90% sparsity
    "wan13b_480p": Workload("wan13b_480p", 1, 12, (21, 30, 52), 128, 64, 1000,
                            "positional", 1),
    # Wan2.1-T2V-14B 720P layer: H40 N75600 (21x45x80), 97% sparsity
    "wan14b_720p": Workload("wan14b_720p", 1, 40, (21, 45, 80), 128, 64, 300,
                            "positional", 2),
    # same shape, fp8 operands, with channel outliers in Q and K
    "wan14b_720p_fp8": Workload("wan14b_720p_fp8", 1, 40, (21, 45, 80), 128, 64, 300,
                                "outliers", 3),
    # same shape with i.i.d. normal Q, K, V: selection without locality, so
    # neighbouring query blocks share few key blocks (a low-reuse bound)
    "wan14b_720p_normal": Workload("wan14b_720p_normal", 1, 40, (21, 45, 80), 128, 64, 300,
                                   "normal", 5),
    # sparsity sweep at the 14B 720P shape with locality + long-range hot blocks
    "sweep": Workload("sweep", 1, 40, (21, 45, 80), 128, 64, 300, "locality", 4,
                      sweep=tuple((b, k) for b in (64, 128)
                                  for k in (300, 1000, 2500, 10000))),
}


def _seed(*parts: int) -> int:
    s = 0x9E3779B97F4A7C15
    for p in parts:
        s = (s * 6364136223846793005 + (int(p) & 0xFFFFFFFF) + 1442695040888963407) % (1 << 63)
    return s


def _gen(*parts: int) -> torch.Generator:
    g = torch.Generator()
    g.manual_seed(_seed(*parts))
    return g


def _coords(grid):
    t, h, w = grid
    tt, yy, xx = torch.meshgrid(torch.arange(t), torch.arange(h), torch.arange(w),
                                indexing="ij")
    return torch.stack([tt.reshape(-1), yy.reshape(-1), xx.reshape(-1)], 1).to(torch.float64)


def _positional(grid, d, g):
    w = torch.randn(d, 3, generator=g, dtype=torch.float64) * 0.25
    phi = torch.rand(d, generator=g, dtype=torch.float64) * (2 * math.pi)
    return math.sqrt(2.0) * torch.sin(_coords(grid) @ w.T + phi)        # [N, d]


def _locality(grid, d, g):
    tau = softmax_scale(d)
    gain = math.sqrt(8.0 / tau)
    w = torch.randn(d, 3, generator=g, dtype=torch.float64) / 3.0
    b = torch.rand(d, generator=g, dtype=torch.float64) * (2 * math.pi)
    p = gain * math.sqrt(2.0 / d) * torch.cos(_coords(grid) @ w.T + b)     # [N, d]
    return p


def _hot_blocks(n, d, g):
    """2% of the 64-token blocks of keys and of queries get one of 8
    orthonormal directions; returns (qadd, kadd) [N, d] float64."""
    nb = -(-n // 64)
    dirs, _ = torch.linalg.qr(torch.randn(d, 8, generator=g, dtype=torch.float64))
    nhot = max(1, round(0.02 * nb))
    kblk = torch.randperm(nb, generator=g)[:nhot]
    qblk = torch.randperm(nb, generator=g)[:nhot]
    kdir = torch.randint(0, 8, (nhot,), generator=g)
    qdir = torch.randint(0, 8, (nhot,), generator=g)
    qadd = torch.zeros(n, d, dtype=torch.float64)
    kadd = torch.zeros(n, d, dtype=torch.float64)
    for blk, di in zip(kblk.tolist(), kdir.tolist()):
        kadd[blk * 64:min(blk * 64 + 64, n)] += dirs[:, di]
    for blk, di in zip(qblk.tolist(), qdir.tolist()):
        qadd[blk * 64:min(blk * 64 + 64, n)] += dirs[:, di]
    return qadd, kadd


def _outlier_pairs(wl: Workload):
    """(head, channel) pairs that carry 20x outliers, for Q and for K."""
    g = _gen(wl.seed, 777)
    npairs = max(1, round(0.001 * wl.heads * wl.head_dim))
    perm_q = torch.randperm(wl.heads * wl.head_dim, generator=g)[:npairs]
    perm_k = torch.randperm(wl.heads * wl.head_dim, generator=g)[:npairs]
    as_pairs = lambda p: [(int(x) // wl.head_dim, int(x) % wl.head_dim) for x in p]
    return as_pairs(perm_q), as_pairs(perm_k)


def make_head(wl: Workload, b: int, h: int):
    """bf16 (q, k, v) of one (batch, head) slice, each [N, d], on the CPU."""
    n, d = wl.seqlen, wl.head_dim
    g = _gen(wl.seed, b, h)
    if wl.gen == "normal":
        q = torch.randn(n, d, generator=g)
        k = torch.randn(n, d, generator=g)
        v = torch.randn(n, d, generator=g)
    elif wl.gen in ("positional", "outliers"):
        p = _positional(wl.grid, d, g).to(torch.float32)
        q = p + 0.5 * torch.randn(n, d, generator=g)
        k = p + 0.5 * torch.randn(n, d, generator=g)
        v = torch.randn(n, d, generator=g)
        if wl.gen == "outliers":
            pq, pk = _outlier_pairs(wl)
            for hh, c in pq:
                if hh == h:
                    q[:, c] *= 20.0
            for hh, c in pk:
                if hh == h:
                    k[:, c] *= 20.0
    elif wl.gen == "locality":
        p = _locality(wl.grid, d, g)
        qadd, kadd = _hot_blocks(n, d, g)
        gain = math.sqrt(8.0 / softmax_scale(d))
        q = (p + gain * qadd).to(torch.float32) + 0.5 * torch.randn(n, d, generator=g)
        k = (p + gain * kadd).to(torch.float32) + 0.5 * torch.randn(n, d, generator=g)
        v = torch.randn(n, d, generator=g)
    else:
        raise ValueError(wl.gen)
    return q.to(torch.bfloat16), k.to(torch.bfloat16), v.to(torch.bfloat16)


def make_inputs(wl: Workload, heads=None):
    """bf16 Q, K, V [B, H', N, d] (CPU) for the listed heads (all by default)."""
    heads = list(range(wl.heads)) if heads is None else list(heads)
    n, d = wl.seqlen, wl.head_dim
    out = [torch.empty(wl.batch, len(heads), n, d, dtype=torch.bfloat16) for _ in range(3)]
    for b in range(wl.batch):
        for hi, h in enumerate(heads):
            for t, x in zip(out, make_head(wl, b, h)):
                t[b, hi] = x
    return tuple(out)


def random_block_lists(nqb: int, nkb: int, kmax: int, seed: int, p_empty: float = 0.05):
    """Random ragged ELL block lists: cnt[i] in [0, kmax] (about p_empty of the
    rows empty), idx[i, :cnt[i]] distinct ascending key blocks, the rest -1."""
    rng = np.random.default_rng(seed)
    idx = np.full((nqb, kmax), -1, dtype=np.int32)
    cnt = rng.integers(1, kmax + 1, size=nqb).astype(np.int32)
    cnt[rng.random(nqb) < p_empty] = 0
    cnt = np.minimum(cnt, nkb)
    for i in range(nqb):
        idx[i, :cnt[i]] = np.sort(rng.choice(nkb, size=cnt[i], replace=False))
    return idx, cnt


# --------------------------------------------------------------------------
# Inputs of the compensation branch: the rotary schedule and synthetic
# low-rank weights (the trained ones are not available).
# --------------------------------------------------------------------------
def rope_pairs_wan(head_dim: int = 128, theta: float = 10000.0):
    """(axis, freq) of every coordinate pair of the 3D RoPE schedule of a
    Wan-style video DiT over head_dim coordinates: a time band of
    head_dim - 4*(head_dim//6) coordinates, then height and width bands of
    2*(head_dim//6) each; in a band of width w the k-th pair turns by
    theta^(-2k/w) radians per grid step along the band's axis."""
    third = head_dim // 6
    axis, freq = [], []
    for ax, w in ((0, head_dim - 4 * third), (1, 2 * third), (2, 2 * third)):
        for k in range(w // 2):
            axis.append(ax)
            freq.append(theta ** (-2.0 * k / w))
    return np.array(axis), np.array(freq)


def rope_table(grid, rank: int, head_dim: int = 128) -> np.ndarray:
    """float32 (cos, sin) [N, rank/2, 2] of the first `rank` coordinates of
    that schedule at every token of the t-major latent grid (T, Hg, Wg)."""
    axis, freq = rope_pairs_wan(head_dim)
    axis, freq = axis[:rank // 2], freq[:rank // 2]
    pos = _coords(grid).numpy()
    ang = pos[:, axis] * freq[None, :]
    return np.ascontiguousarray(np.stack([np.cos(ang), np.sin(ang)], axis=-1), dtype=np.float32)


def comp_params(wl: Workload, rank: int = 64, gate_scale: float = 0.5, seed_extra: int = 0):
    """Synthetic compensation-branch inputs of a workload: low-rank
    projections P_q, P_k bf16 [H, rank, d] ~ N(0, 1/d), RMSNorm weights
    gamma fp32 [H, d] ~ 1 + 0.1 N(0, 1), token-wise gates fp32 [B, H, N]
    ~ gate_scale * N(0, 1)."""
    g = _gen(wl.seed, 991, seed_extra)
    d = wl.head_dim
    pq = (torch.randn(wl.heads, rank, d, generator=g) / math.sqrt(d)).to(torch.bfloat16)
    pk = (torch.randn(wl.heads, rank, d, generator=g) / math.sqrt(d)).to(torch.bfloat16)
    gamma = 1.0 + 0.1 * torch.randn(wl.heads, d, generator=g)
    gate = gate_scale * torch.randn(wl.batch, wl.heads, wl.seqlen, generator=g)
    return pq, pk, gamma, gate


# --------------------------------------------------------------------------
# Inputs of the W8A8 linear layers: activations with channel outliers and
# synthetic weights (the trained ones are not available).
# --------------------------------------------------------------------------
# (tokens M, in features K, out features N) of the 14B-720P block's linears:
# the q/k/v/o projections and the two feed-forward layers (hidden 5120,
# FFN 13824), at 75,600 tokens.
LINEAR_SHAPES = {
    "wan14b_720p_qkvo": (75600, 5120, 5120),
    "wan14b_720p_ffn_up": (75600, 5120, 13824),
    "wan14b_720p_ffn_down": (75600, 13824, 5120),
}


def linear_inputs(m: int, k: int, n: int, seed: int = 0, outlier_frac: float = 0.001,
                  outlier_gain: float = 20.0, rows=None):
    """bf16 activations X [M', K] and weights W [N, K], fp32 bias [N].

    X ~ N(0, 1) with a fraction ``outlier_frac`` of the input channels (at
    least one) multiplied by ``outlier_gain`` on every token, as the channel
    outliers of transformer activations; each token also gets a gain
    exp(0.5 N(0, 1)) so per-token scales differ.  W ~ N(0, 1/K) with a
    per-output-channel gain exp(0.5 N(0, 1)); bias ~ 0.1 N(0, 1).  Every
    token row is drawn from its own seed, so ``rows`` (a list of token
    indices) regenerates just those rows."""
    gw = _gen(seed, 4242)
    w = torch.randn(n, k, generator=gw) / math.sqrt(k)
    w = (w * torch.exp(0.5 * torch.randn(n, 1, generator=gw))).to(torch.bfloat16)
    bias = 0.1 * torch.randn(n, generator=gw)
    n_out = max(1, int(round(outlier_frac * k)))
    ch = torch.randperm(k, generator=gw)[:n_out]
    chan_gain = torch.ones(k)
    chan_gain[ch] = outlier_gain
    step = 256                                   # token rows drawn per generator
    rows = list(range(m)) if rows is None else list(rows)
    x = torch.empty(len(rows), k, dtype=torch.bfloat16)
    by_chunk = {}
    for i, r in enumerate(rows):
        if not 0 <= r < m:
            raise IndexError(r)
        by_chunk.setdefault(r // step, []).append((i, r))
    for c, members in by_chunk.items():
        g = _gen(seed, 4243, c)
        lo, hi = c * step, min(m, (c + 1) * step)
        xc = torch.randn(hi - lo, k, generator=g)
        xc = (xc * torch.exp(0.5 * torch.randn(hi - lo, 1, generator=g)) * chan_gain).to(torch.bfloat16)
        dst = torch.tensor([i for i, _ in members])
        src = torch.tensor([r - lo for _, r in members])
        x[dst] = xc[src]
    return x, w, bias

"""Shared plumbing of the GPU parity tests: seeded inputs, oracle per head,
error metrics.  (Not a test module.)"""
import sys

import numpy as np
import torch

import oracle as O

# Parity bar: index lists bit-exact; bf16 outputs rel-L2 <= 1e-2 and max-abs
# <= 2e-2 against the fp64 oracle; fp8 outputs rel-L2 <= 5e-2.
BF16_REL_L2 = 1e-2
BF16_MAX_ABS = 2e-2
FP8_REL_L2 = 5e-2
LSE_ABS = 2e-3
# fp8 path: the row sum is taken over the probabilities rounded to e4m3
# (nearest even, 3 mantissa bits), each within a relative 2^-4 of its exact
# value, so the sum (and exp(LSE)) is within a relative 2^-4 as well and LSE
# within log(1 + 2^-4); 2e-3 more covers the fp32 arithmetic.
FP8_LSE_ABS = float(np.log1p(2.0 ** -4)) + 2e-3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def widen(t):
    """bf16 CPU tensor -> float64 numpy (exact)."""
    return t.to(torch.float64).numpy()


def rel_l2(x, ref):
    ref = np.asarray(ref, dtype=np.float64)
    x = np.asarray(x, dtype=np.float64)
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(x - ref) / (den if den > 0 else 1.0))


def oracle_select(q, k, block, keep_bp, mode="row"):
    """q, k: bf16 CPU [N, d] -> (idx, cnt) of the oracle."""
    return O.select_head(widen(q), widen(k), block, keep_bp, mode)


def oracle_attend(q, k, v, idx, cnt, block, tau, qblocks=None):
    return O.sparse_attention(widen(q), widen(k), widen(v), idx, cnt, block, tau, qblocks)


def check_out(o_gpu, lse_gpu, o_ref, lse_ref, rows=None, rel=BF16_REL_L2, mabs=BF16_MAX_ABS,
              what=""):
    """o_gpu [N, d] (any float dtype, CPU), lse_gpu [N] against the oracle."""
    o = o_gpu.to(torch.float64).numpy()
    lse = lse_gpu.to(torch.float64).numpy() if lse_gpu is not None else None
    if rows is not None:
        o, o_ref = o[rows], o_ref[rows]
        lse = lse[rows] if lse is not None else None
        lse_ref = lse_ref[rows]
    err = rel_l2(o, o_ref)
    mx = float(np.abs(o - o_ref).max()) if o.size else 0.0
    say(f"  {what}: rel_l2={err:.3e} max_abs={mx:.3e}")
    assert err <= rel, (what, err)
    if mabs is not None:
        assert mx <= mabs, (what, mx)
    if lse is not None:
        fin = np.isfinite(lse_ref)
        assert np.array_equal(np.isneginf(lse), np.isneginf(lse_ref)), what
        if fin.any():
            assert np.abs(lse[fin] - lse_ref[fin]).max() <= LSE_ABS, what


# ---- the library's launch order (its own definition, stated in the header of
# sparse_attn_schedule; the paper fixes no order: only performance depends on
# it) -------------------------------------------------------------------------
XCD_RUN, XCDS = 256, 8


def sorted_position(s, G):
    """Sorted position taken by launch slot s of G (runs of 256 per XCD)."""
    group = XCDS * XCD_RUN
    if s >= (G // group) * group:
        return s
    return group * (s // group) + XCD_RUN * (s % XCDS) + (s % group) // XCDS


def tile_classes(cnt, kmax, seqlen, block):
    """Cost class of every query tile t = (b*H + h) * ceil(L/64) + row/64."""
    cnt = np.asarray(cnt)
    B, H, nb = cnt.shape
    ntiles = -(-seqlen // 64)
    t = np.arange(B * H * ntiles)
    bh, qt = t // ntiles, t % ntiles
    c = np.clip(cnt.reshape(-1)[bh * nb + (qt * 64) // block], 0, kmax)
    tiles = c * (block // 64)
    bits = np.zeros_like(tiles)
    nz = tiles > 0
    bits[nz] = np.floor(np.log2(tiles[nz])).astype(np.int64) + 1
    return np.minimum(bits, 15)


def check_launch_order(order, cnt, kmax, seqlen, block, what=""):
    """Properties of a launch order: a permutation of every query tile; read
    back in sorted position (the XCD interleave undone), cost classes do not
    increase, and tiles of one class keep raster order."""
    order = np.asarray(order, dtype=np.int64)
    G = order.size
    assert np.array_equal(np.sort(order), np.arange(G)), (what, "not a permutation")
    pos = np.array([sorted_position(s, G) for s in range(G)], dtype=np.int64)
    seq = np.empty(G, dtype=np.int64)
    seq[pos] = order
    cls = tile_classes(cnt, kmax, seqlen, block)[seq]
    assert np.all(np.diff(cls) <= 0), (what, "classes increase along sorted positions")
    same = np.diff(cls) == 0
    assert np.all(np.diff(seq)[same] > 0), (what, "equal classes out of raster order")


def fp8_tiles_to_rows(x8t, N, operand):
    """Invert the K (operand 0) or V (operand 1) tile layout of
    sparse_attn_quant_fp8_tiles: uint8 [B, H, T, 8192] -> ([B, H, N, 128]
    row-major codes, the codes of the T*64 - N keys past N).  Only index
    arithmetic: the layout formulas of the header, read backwards."""
    x = np.asarray(x8t)
    B, H, T, _ = x.shape
    c = np.arange(512)[:, None]
    e = np.arange(16)[None, :]
    f, lane = c // 64, c % 64
    l, g = lane % 32, lane // 32
    if operand == 0:
        rt, ks, hf = f // 4, (f // 2) % 2, f % 2
        key, ch = 32 * rt + l + 0 * e, 64 * ks + 32 * g + 16 * hf + e
    else:
        dt, hf = f // 2, f % 2
        key, ch = 32 * hf + 8 * (e // 4) + 4 * g + e % 4, 32 * dt + l + 0 * e
    rows = np.zeros((B, H, T, 64, 128), dtype=np.uint8)
    rows[:, :, :, key, ch] = x.reshape(B, H, T, 512, 16)
    rows = rows.reshape(B, H, T * 64, 128)
    return rows[:, :, :N], rows[:, :, N:]

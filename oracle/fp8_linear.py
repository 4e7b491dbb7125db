"""W8A8 FP8 (E4M3) linear layer, written out from its definition (test
infrastructure only; the product path never imports this package).

Paper §4.3 (FP8 quantization): the linear projections of attention and the
feed-forward layers run as W8A8 FP8 E4M3; each weight output channel has a
static scale fixed once offline, each activation token a scale computed at
run time, and the per-token activation quantisation is a single fused pass
(scale and cast together).  Normalisation, gating and mask selection stay in
BF16, so the layer's output is bf16.

Readings where the paper is silent (stated in the design notes):
  * One scale per row (token of the activations, output channel of the
    weights): a = max |x| over the row (bf16 values, exact in fp32), floored
    at 2^-100 so that its reciprocal stays a finite fp32; the scale is
    s = fp32(a / 448) and the codes are e4m3(fp32(x * fp32(448 / a))),
    rounded to nearest with ties to even.  These fp32 roundings decide the
    codes, so they are taken in fp32 here too (numpy float32 arithmetic is
    IEEE-754 binary32 with round-to-nearest-even); 448 is the largest e4m3
    magnitude, so the row maximum lands on it.
  * y[m, n] = (sum_k dec(a8[m, k]) * dec(w8[n, k])) * s_a[m] * s_w[n]
    (+ bias[n]), evaluated in fp64 here and rounded to bf16 by the product.
"""
from __future__ import annotations

import numpy as np

from .sparse_attention import E4M3_MAX, e4m3_encode, e4m3_table

__all__ = ["ROW_AMAX_FLOOR", "quant_rows_fp8", "dequant_rows_fp8", "linear_w8a8"]

ROW_AMAX_FLOOR = 2.0 ** -100


def quant_rows_fp8(x):
    """Per-row E4M3 quantisation of x [R, C] (values exact in fp32, e.g. bf16
    widened).  Returns (codes uint8 [R, C], scales float32 [R])."""
    x32 = np.asarray(x, dtype=np.float32)
    if x32.ndim != 2:
        raise ValueError("x must be 2-D")
    amax = np.max(np.abs(x32), axis=1) if x32.shape[1] else np.zeros(x32.shape[0], np.float32)
    amax = np.maximum(amax, np.float32(ROW_AMAX_FLOOR))
    fmax = np.float32(E4M3_MAX)
    scale = (amax / fmax).astype(np.float32)           # fp32 quotient
    inv = (fmax / amax).astype(np.float32)             # fp32 quotient
    y = (x32 * inv[:, None]).astype(np.float32)        # fp32 product
    codes = e4m3_encode(y.astype(np.float64))
    return codes, scale


def dequant_rows_fp8(codes, scale):
    """dec(code) * s of the row, in fp64."""
    return e4m3_table()[np.asarray(codes).astype(np.int64)] * np.asarray(scale, np.float64)[:, None]


def linear_w8a8(a8, sa, w8, sw, bias=None):
    """y [M, N] = (A W^T) * s_a s_w^T (+ bias) over the decoded codes, fp64."""
    table = e4m3_table()
    a = table[np.asarray(a8).astype(np.int64)]
    w = table[np.asarray(w8).astype(np.int64)]
    y = (a @ w.T) * np.asarray(sa, np.float64)[:, None] * np.asarray(sw, np.float64)[None, :]
    if bias is not None:
        y = y + np.asarray(bias, np.float64)[None, :]
    return y

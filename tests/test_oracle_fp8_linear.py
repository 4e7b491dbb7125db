"""Pins of the oracle's W8A8 FP8 linear layer (paper §4.3) against facts
independent of it: a library fp8 cast, the row maximum landing on 448,
power-of-two scale equivariance, the e4m3 rounding bound, a brute-force
product with exact summation, and the end-to-end quantisation error bound
against the unquantised product."""
import math

import numpy as np
import torch

import oracle as O
import workloads as W


def _bf16(a):
    return torch.from_numpy(np.asarray(a, np.float32)).to(torch.bfloat16).float().numpy()


def test_codes_match_library_cast_of_the_scaled_row():
    x, _, _ = W.linear_inputs(300, 1024, 8, seed=3)
    x = x.float().numpy()
    codes, scale = O.quant_rows_fp8(x)
    # the scaled value in fp32 arithmetic, cast by torch's e4m3fn conversion
    amax = np.abs(x).max(axis=1).astype(np.float32)
    inv = np.float32(448.0) / amax
    y = torch.from_numpy((x * inv[:, None]).astype(np.float32))
    ref = y.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(codes, ref)
    assert np.array_equal(scale, (amax / np.float32(448.0)).astype(np.float32))


def test_row_maximum_lands_on_448_and_zero_rows():
    rng = np.random.default_rng(1)
    x = _bf16(rng.standard_normal((50, 96)) * rng.uniform(1e-3, 1e3, (50, 1)))
    codes, scale = O.quant_rows_fp8(x)
    j = np.argmax(np.abs(x), axis=1)
    top = codes[np.arange(50), j]
    assert np.all((top & 0x7F) == 0x7E)                     # |448|
    assert np.all((top >> 7) == (x[np.arange(50), j] < 0))  # sign kept
    z, sz = O.quant_rows_fp8(np.zeros((2, 16)))
    assert np.all((z & 0x7F) == 0)
    assert np.all(sz == np.float32(2.0 ** -100 / 448.0))
    assert np.all(np.isfinite(sz)) and np.all(sz > 0)


def test_power_of_two_scale_equivariance():
    """Multiplying a row by 2^j (exact in bf16) leaves its codes unchanged and
    multiplies its scale by 2^j: every fp32 step commutes with it."""
    rng = np.random.default_rng(2)
    x = _bf16(rng.standard_normal((20, 64)))
    c0, s0 = O.quant_rows_fp8(x)
    for j in (-20, -3, 5, 40):
        c1, s1 = O.quant_rows_fp8(x * 2.0 ** j)
        assert np.array_equal(c0, c1)
        assert np.array_equal(s1, (s0 * np.float32(2.0 ** j)).astype(np.float32))


def test_rounding_error_bound():
    """|dec(code) s - x| <= 2^-4 |x| (half an e4m3 mantissa step) plus half
    the subnormal step 2^-10 s, plus the fp32 roundings of s, 448/a and the
    product (a few 2^-24 relative)."""
    x, _, _ = W.linear_inputs(200, 2048, 8, seed=4)
    x = x.float().numpy().astype(np.float64)
    codes, scale = O.quant_rows_fp8(x)
    err = np.abs(O.dequant_rows_fp8(codes, scale) - x)
    bound = (2.0 ** -4 + 4 * 2.0 ** -24) * np.abs(x) + 2.0 ** -10 * scale[:, None].astype(np.float64)
    assert np.all(err <= bound)
    # and the bound is attained to within a factor ~1 (the rounding is nearest, not truncation)
    assert np.max(err / bound) > 0.9


def test_linear_brute_force_exact_sums():
    rng = np.random.default_rng(5)
    a8 = rng.integers(0, 256, (3, 16)).astype(np.uint8)
    w8 = rng.integers(0, 256, (4, 16)).astype(np.uint8)
    a8[(a8 & 0x7F) == 0x7F] = 0x10                          # no NaN codes
    w8[(w8 & 0x7F) == 0x7F] = 0x22
    sa = np.float32([0.5, 3.0, 1e-3])
    sw = np.float32([2.0, 0.25, 7.0, 1.0])
    bias = np.array([0.1, -0.2, 0.0, 5.0])
    y = O.linear_w8a8(a8, sa, w8, sw, bias)

    def dec(c):                       # e4m3fn by its field definition
        s = -1.0 if c & 0x80 else 1.0
        e, f = (c >> 3) & 15, c & 7
        return s * (f / 8.0) * 2.0 ** -6 if e == 0 else s * (1 + f / 8.0) * 2.0 ** (e - 7)

    for m in range(3):
        for n in range(4):
            acc = math.fsum(dec(int(a8[m, k])) * dec(int(w8[n, k])) for k in range(16))
            ref = acc * float(sa[m]) * float(sw[n]) + bias[n]
            assert math.isclose(y[m, n], ref, rel_tol=1e-14, abs_tol=1e-14)


def test_end_to_end_error_bound_against_unquantised_product():
    """|y_q - x w^T| <= sum_k |x_k w_k| ((1 + e)^2 - 1) + subnormal terms,
    e = 2^-4 + 2^-22, from the per-element bound of both operands."""
    x, w, bias = W.linear_inputs(64, 1024, 48, seed=6)
    x = x.float().numpy().astype(np.float64)
    w = w.float().numpy().astype(np.float64)
    a8, sa = O.quant_rows_fp8(x)
    w8, sw = O.quant_rows_fp8(w)
    y = O.linear_w8a8(a8, sa, w8, sw, bias.numpy())
    exact = x @ w.T + bias.numpy()[None, :]
    e = 2.0 ** -4 + 2.0 ** -22
    absprod = np.abs(x) @ np.abs(w).T
    # subnormal halves: 2^-10 s on each side times the other operand's magnitude (+ their product)
    ta = 2.0 ** -10 * sa[:, None].astype(np.float64) * np.abs(w).sum(1)[None, :] * (1 + e)
    tw = 2.0 ** -10 * sw[None, :].astype(np.float64) * np.abs(x).sum(1)[:, None] * (1 + e)
    tt = 2.0 ** -20 * sa[:, None].astype(np.float64) * sw[None, :] * x.shape[1]
    bound = absprod * ((1 + e) ** 2 - 1) + ta + tw + tt
    assert np.all(np.abs(y - exact) <= bound)
    # the layer is close on average: per-token relative L2 error of a few percent at most
    rel = np.linalg.norm(y - exact) / np.linalg.norm(exact)
    assert rel < 0.05, rel


def test_identity_weight_returns_dequantised_activations():
    """W = I (exact in e4m3 with scale 1/448 * 448): y = dec(a8) s_a."""
    rng = np.random.default_rng(7)
    x = _bf16(rng.standard_normal((5, 32)))
    a8, sa = O.quant_rows_fp8(x)
    w8, sw = O.quant_rows_fp8(np.eye(32))
    assert np.all(sw == np.float32(1.0 / 448.0))
    y = O.linear_w8a8(a8, sa, w8, sw)
    ref = O.dequant_rows_fp8(a8, sa)
    assert np.allclose(y, ref * (448.0 * np.float64(np.float32(1.0 / 448.0))), rtol=1e-15, atol=0)

"""Pins of the fp64 oracle against facts that do not come from the oracle
itself: hand-computed fixtures, closed forms, brute force on tiny inputs,
library routines for the special cases that reduce to them, and invariants.
CPU only."""
import itertools
import math
import os

import numpy as np
import pytest
import torch

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TAU = float(np.float32(1.0 / math.sqrt(128)))


def rnd(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


# ----------------------------------------------------------------- partition
def test_block_partition_and_keep_count():
    assert O.block_sizes(4096, 64).tolist() == [64] * 64
    s = O.block_sizes(75600, 64)
    assert s.size == 1182 and s[-1] == 16 and s[:-1].min() == 64
    s = O.block_sizes(32760, 64)
    assert s.size == 512 and s[-1] == 56
    s = O.block_sizes(75600, 128)
    assert s.size == 591 and s[-1] == 80
    # keep ratio -> k: ceil in integers (10% of 64 blocks keeps 7)
    assert O.keep_count(1000, 64) == 7
    assert O.keep_count(300, 1182) == 36
    assert O.keep_count(1000, 512) == 52
    assert O.keep_count(1000, 1182) == 119
    assert O.keep_count(2500, 1182) == 296
    assert O.keep_count(300, 591) == 18
    assert O.keep_count(2500, 591) == 148
    assert O.keep_count(10000, 591) == 591
    assert O.keep_count(1, 10) == 1          # clamps to >= 1
    assert O.keep_count(20000, 10) == 10     # clamps to <= nkb


# -------------------------------------------------------------------- scores
def test_scores_equal_bruteforce_block_mean_of_logits():
    # blocks of 8 over N=37 (tail of 5) and keys N=29 (tail of 5)
    q, k = rnd((37, 6), 1), rnd((29, 6), 2)
    s = O.block_scores(q, k, 8)
    assert s.shape == (5, 4)
    for i in range(5):
        for j in range(4):
            tot, cnt = 0.0, 0
            for t in range(i * 8, min(i * 8 + 8, 37)):
                for u in range(j * 8, min(j * 8 + 8, 29)):
                    tot += sum(q[t, c] * k[u, c] for c in range(6))
                    cnt += 1
            assert s[i, j] == pytest.approx(tot / cnt, rel=1e-12, abs=1e-12)


def test_pool_is_exact_for_bf16_inputs():
    # 64 bf16 values with a modest exponent spread sum exactly in fp64:
    # compare against exact rational arithmetic.
    from fractions import Fraction
    bits = torch.randn(64, 4).to(torch.bfloat16)
    x = bits.to(torch.float64).numpy()
    pooled = O.pool_blocks(x, 64)[0]
    for c in range(4):
        exact = sum(Fraction(float(v)) for v in x[:, c])
        assert Fraction(float(pooled[c])) == exact


# --------------------------------------------------------------------- top-k
def _read_topk_cases():
    cases, cur, mode = [], None, None
    with open(os.path.join(GOLDEN, "topk_toy.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("case"):
                _, name, kk = line.split()
                cur = {"name": name, "k": int(kk.split("=")[1]), "s": [], "e": []}
                cases.append(cur)
                mode = "s"
            elif line == "expect":
                mode = "e"
            elif mode == "s":
                cur["s"].append([float(t) for t in line.split()])
            else:
                cur["e"].append([int(t) for t in line.split()])
    return cases


@pytest.mark.parametrize("case", _read_topk_cases(), ids=lambda c: c["name"])
def test_topk_hand_computed(case):
    s = np.array(case["s"])
    got = O.select_row_topk(s, case["k"])
    assert got.tolist() == case["e"]


def _bruteforce_topk(row, k):
    """The unique k-subset S with: every a in S beats every b not in S under
    (score desc, index asc)."""
    n = len(row)
    found = []
    for sub in itertools.combinations(range(n), k):
        rest = [b for b in range(n) if b not in sub]
        if all(row[a] > row[b] or (row[a] == row[b] and a < b) for a in sub for b in rest):
            found.append(list(sub))
    assert len(found) == 1
    return found[0]


def test_topk_bruteforce_with_many_ties():
    rng = np.random.default_rng(5)
    for trial in range(200):
        n = int(rng.integers(1, 9))
        k = int(rng.integers(1, n + 1))
        row = rng.integers(-3, 4, size=n).astype(np.float64)   # many ties
        assert O.topk_ascending(row, k).tolist() == _bruteforce_topk(row, k)


def test_head_topk_hand_computed():
    with open(os.path.join(GOLDEN, "head_topk_toy.txt")) as f:
        lines = [l.strip() for l in f if l.strip() and not l.startswith("#")]
    keep_bp = int(lines[0].split("=")[1])
    e = lines.index("expect")
    s = np.array([[float(t) for t in l.split()] for l in lines[1:e]])
    expect = [[int(t) for t in l.split()] for l in lines[e + 1:]]
    idx, cnt = O.select_head_topk(s, keep_bp)
    assert cnt.tolist() == [len(r) for r in expect]
    for i, r in enumerate(expect):
        assert idx[i, :cnt[i]].tolist() == r
        assert (idx[i, cnt[i]:] == -1).all()


def test_head_topk_invariants():
    rng = np.random.default_rng(9)
    s = rng.integers(-5, 6, size=(7, 9)).astype(np.float64)
    idx, cnt = O.select_head_topk(s, 3000)
    total = -(-3000 * 63 // 10000)
    assert cnt.sum() == total and cnt.min() >= 1
    chosen = np.zeros_like(s, dtype=bool)
    for i in range(7):
        chosen[i, idx[i, :cnt[i]]] = True
        assert chosen[i, O.topk_ascending(s[i], 1)[0]]
    # every extra pair beats every unchosen pair under (s desc, i asc, j asc)
    top1 = {(i, int(O.topk_ascending(s[i], 1)[0])) for i in range(7)}
    extra = [(i, j) for i in range(7) for j in range(9) if chosen[i, j] and (i, j) not in top1]
    unchosen = [(i, j) for i in range(7) for j in range(9) if not chosen[i, j]]
    key = lambda p: (-s[p], p[0], p[1])
    assert max(key(p) for p in extra) < min(key(p) for p in unchosen)


def test_head_topk_rows_are_row_prefixes_and_cap():
    """Each row's ragged selection is the row's own top-cnt_i under
    (score desc, j asc) -- the property the GPU path reduces the mode to --
    and a row stride kmax keeps the kmax best of a longer row."""
    rng = np.random.default_rng(11)
    for trial in range(20):
        nqb, nkb = rng.integers(2, 9), rng.integers(2, 11)
        s = rng.integers(-4, 5, size=(nqb, nkb)).astype(np.float64)   # many ties
        budget = int(rng.integers(nqb, nqb * nkb + 1))
        idx, cnt = O.select_head_topk(s, budget=budget)
        assert cnt.sum() == budget
        for i in range(nqb):
            assert idx[i, :cnt[i]].tolist() == O.topk_ascending(s[i], int(cnt[i])).tolist()
        kmax = int(rng.integers(1, nkb + 1))
        ci, cc = O.select_head_topk(s, budget=budget, kmax=kmax)
        assert ci.shape == (nqb, kmax)
        assert cc.tolist() == np.minimum(cnt, kmax).tolist()
        for i in range(nqb):
            assert ci[i, :cc[i]].tolist() == O.topk_ascending(s[i], int(cc[i])).tolist()
            assert (ci[i, cc[i]:] == -1).all()
    # budget from a keep ratio
    assert O.head_pair_budget(3000, 7, 9) == 19
    assert O.head_pair_budget(1, 7, 9) == 7
    assert O.head_pair_budget(10000, 7, 9) == 63


# ----------------------------------------------------------------- attention
def _dense_sdpa(q, k, v, tau):
    qt, kt, vt = (torch.from_numpy(x)[None, None] for x in (q, k, v))
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=tau)
    return o[0, 0].numpy()


def test_keep_all_equals_dense_attention_library():
    n, d, b = 200, 32, 16                 # 13 blocks, tail of 8
    q, k, v = rnd((n, d), 11), rnd((n, d), 12), rnd((n, d), 13)
    idx, cnt = O.select_head(q, k, b, 10000)
    assert (cnt == 13).all() and (idx == np.arange(13)).all()
    out, lse = O.sparse_attention(q, k, v, idx, cnt, b, TAU)
    np.testing.assert_allclose(out, _dense_sdpa(q, k, v, TAU), rtol=1e-12, atol=1e-12)
    ref_lse = torch.logsumexp(torch.from_numpy(TAU * (q @ k.T)), dim=1).numpy()
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-13, atol=1e-13)


def test_explicit_mask_bruteforce():
    n, d, b, tau = 37, 5, 8, 0.7        # 5 query/key blocks, tail of 5
    q, k, v = rnd((n, d), 21), rnd((n, d), 22), rnd((n, d), 23)
    idx, cnt = O.select_head(q, k, b, 4000)       # k = 2 of 5
    out, lse = O.sparse_attention(q, k, v, idx, cnt, b, tau)
    for t in range(n):
        allowed = set(idx[t // b, :cnt[t // b]].tolist())
        z = [tau * sum(q[t, c] * k[u, c] for c in range(d)) if u // b in allowed else -math.inf
             for u in range(n)]
        m = max(z)
        w = [math.exp(x - m) if x != -math.inf else 0.0 for x in z]
        tot = sum(w)
        for c in range(d):
            assert out[t, c] == pytest.approx(sum(w[u] * v[u, c] for u in range(n)) / tot,
                                              rel=1e-11, abs=1e-12)
        assert lse[t] == pytest.approx(m + math.log(tot), rel=1e-12, abs=1e-12)


def test_probabilities_are_row_stochastic_and_confined():
    # V = identity turns O into the probability matrix itself.
    n, b = 48, 8                          # 6 blocks
    q, k = rnd((n, 16), 31, 2.0), rnd((n, 16), 32, 2.0)
    v = np.eye(n)
    idx, cnt = O.select_head(q, k, b, 5000)      # 3 of 6
    p, _ = O.sparse_attention(q, k, v, idx, cnt, b, TAU)
    assert (p >= 0).all()
    np.testing.assert_allclose(p.sum(axis=1), 1.0, atol=1e-13)
    for t in range(n):
        allowed = np.zeros(n, dtype=bool)
        for j in idx[t // b]:
            allowed[j * b:(j + 1) * b] = True
        assert (p[t, ~allowed] == 0).all() and (p[t, allowed] > 0).all()


def test_constant_values_give_constant_output():
    n, d, b = 100, 8, 16
    q, k = rnd((n, d), 41), rnd((n, d), 42)
    v = np.tile(np.linspace(-2, 3, d), (n, 1))
    idx, cnt = O.select_head(q, k, b, 3000)
    out, _ = O.sparse_attention(q, k, v, idx, cnt, b, TAU)
    np.testing.assert_allclose(out, v, rtol=0, atol=1e-13)


def test_zero_queries_closed_form():
    # Q = 0: every score is 0, ties keep blocks 0..k-1, and every logit is 0,
    # so O_t is the plain mean of v over the first k key blocks; LSE = log n.
    n, d, b = 90, 6, 16                   # 6 blocks, tail of 10
    q = np.zeros((n, d))
    k, v = rnd((n, d), 51), rnd((n, d), 52)
    idx, cnt = O.select_head(q, k, b, 5000)      # k = 3
    assert (idx == np.arange(3)).all()
    out, lse = O.sparse_attention(q, k, v, idx, cnt, b, TAU)
    np.testing.assert_allclose(out, np.tile(v[:48].mean(axis=0), (n, 1)), atol=1e-14)
    np.testing.assert_allclose(lse, math.log(48), atol=1e-14)


def test_key_block_permutation_invariance():
    n, d, b = 96, 8, 16                   # 6 full blocks
    q, k, v = rnd((n, d), 61), rnd((n, d), 62), rnd((n, d), 63)
    idx, cnt = O.select_head(q, k, b, 5000)
    out, lse = O.sparse_attention(q, k, v, idx, cnt, b, TAU)
    perm = np.array([3, 0, 5, 1, 4, 2])             # new block p holds old block perm[p]
    rows = np.concatenate([np.arange(j * b, (j + 1) * b) for j in perm])
    idx2, cnt2 = O.select_head(q, k[rows], b, 5000)
    inv = np.argsort(perm)
    assert [sorted(perm[r].tolist()) for r in idx2] == [r.tolist() for r in idx]
    assert [sorted(inv[r].tolist()) for r in idx] == [r.tolist() for r in idx2]
    out2, lse2 = O.sparse_attention(q, k[rows], v[rows], idx2, cnt2, b, TAU)
    np.testing.assert_allclose(out2, out, atol=1e-13)
    np.testing.assert_allclose(lse2, lse, atol=1e-13)


def test_single_block_is_dense():
    n, d = 50, 16
    q, k, v = rnd((n, d), 71), rnd((n, d), 72), rnd((n, d), 73)
    idx, cnt = O.select_head(q, k, 64, 300)
    assert idx.tolist() == [[0]]
    out, _ = O.sparse_attention(q, k, v, idx, cnt, 64, TAU)
    np.testing.assert_allclose(out, _dense_sdpa(q, k, v, TAU), rtol=1e-12, atol=1e-12)


def test_empty_rows():
    n, d, b = 40, 4, 8
    q, k, v = rnd((n, d), 81), rnd((n, d), 82), rnd((n, d), 83)
    idx = np.array([[1, 3], [-1, -1], [0, -1], [-1, -1], [4, -1]], dtype=np.int32)
    cnt = np.array([2, 0, 1, 0, 1], dtype=np.int32)
    out, lse = O.sparse_attention(q, k, v, idx, cnt, b, TAU)
    assert (out[8:16] == 0).all() and np.isneginf(lse[8:16]).all()
    assert (out[24:32] == 0).all() and np.isneginf(lse[24:32]).all()
    assert np.isfinite(lse[:8]).all()


def test_sampled_rows_match_full():
    n, d, b = 130, 8, 16
    q, k, v = rnd((n, d), 91), rnd((n, d), 92), rnd((n, d), 93)
    idx, cnt = O.select_head(q, k, b, 3000)
    out, lse = O.sparse_attention(q, k, v, idx, cnt, b, TAU)
    out2, lse2 = O.sparse_attention(q, k, v, idx, cnt, b, TAU, qblocks=[0, 8])
    np.testing.assert_array_equal(out2[:16], out[:16])
    np.testing.assert_array_equal(out2[128:], out[128:])


# ----------------------------------------------------------------------- fp8
def test_e4m3_table_matches_library():
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    t = O.e4m3_table()
    assert np.array_equal(np.isnan(t), np.isnan(ref))
    assert np.array_equal(t[~np.isnan(t)], ref[~np.isnan(ref)])
    assert t[0x7E] == 448.0 and t[0x01] == 2.0 ** -9 and t[0x08] == 2.0 ** -6


def test_e4m3_encode_matches_library_in_range():
    x = np.concatenate([rnd(200000, 3, 50.0), rnd(20000, 4, 1e-3), rnd(20000, 5, 1e-2)])
    x = np.clip(x, -448, 448)
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(O.e4m3_encode(x), ref)


def test_e4m3_encode_ties_saturation_roundtrip():
    enc = lambda v: int(O.e4m3_encode(np.array([v]))[0])
    assert enc(1.0625) == 0x38          # tie 1.0 | 1.125 -> even (1.0)
    assert enc(1.1875) == 0x3A          # tie 1.125 | 1.25 -> even (1.25)
    assert enc(2.0 ** -10) == 0x00      # tie 0 | 2^-9 -> even (0)
    assert enc(3 * 2.0 ** -10) == 0x02  # tie 2^-9 | 2^-8 -> even (2^-8)
    assert enc(-0.0) == 0x80 and enc(-(2.0 ** -11)) == 0x80
    assert enc(500.0) == 0x7E and enc(-1e9) == 0xFE and enc(448.0) == 0x7E
    assert enc(464.0) == 0x7E           # halfway to the (absent) 480 saturates
    t = O.e4m3_table()
    for c in list(range(0, 127)) + list(range(128, 255)):
        assert enc(t[c]) == c


def test_fp8_scale_exponent_bruteforce():
    vals = [448.0, 447.0, 449.0, 224.0, 224.0000001, 1.0, 3.5, 1e-6, 123456.0,
            np.nextafter(448.0, 0), np.nextafter(448.0, 1e9), 448.0 * 2 ** -20,
            np.nextafter(448.0 * 2 ** -20, 1.0)]
    vals += list(rnd(300, 7, 30.0).__abs__())
    for a in vals:
        e = O.fp8_scale_exponent(float(a))
        brute = next(ee for ee in range(-200, 200) if a <= 448.0 * 2.0 ** ee)
        assert e == max(brute, -126), a
    assert O.fp8_scale_exponent(0.0) == 0
    assert O.fp8_scale_exponent(1e-40) == -126          # clamped: 2^e stays a normal fp32


def test_quantize_blocks_properties():
    x = np.concatenate([rnd((64, 16), 8, 3.0), rnd((64, 16), 9, 0.01), rnd((10, 16), 10, 100.0)])
    codes, scales = O.quantize_fp8_blocks(x, 64)
    assert scales.size == 3
    t = O.e4m3_table()
    for i, sc in enumerate(scales):
        rows = slice(i * 64, min(i * 64 + 64, x.shape[0]))
        assert math.log2(sc) == int(math.log2(sc))              # a power of two
        amax = np.abs(x[rows]).max() / sc
        assert 224.0 < amax <= 448.0                             # top binade used
        xr = x[rows] / sc
        dec = t[codes[rows].astype(int)]
        # nearest-rounding bound: half a spacing of the binade (or subnormal spacing)
        spacing = np.maximum(2.0 ** (np.floor(np.log2(np.maximum(np.abs(xr), 2.0 ** -6))) - 3),
                             2.0 ** -9)
        assert (np.abs(dec - xr) <= spacing / 2 + 1e-300).all()
    deq = O.dequantize_fp8_blocks(codes, scales, 64)
    assert np.abs(deq - x).max() <= 0.07 * np.abs(x).max()


def test_fp8_path_is_exact_on_representable_inputs():
    # inputs already on the e4m3 grid of their block scale: quantisation is
    # the identity, so the fp8 path equals the plain path bit for bit.
    t = O.e4m3_table()
    rng = np.random.default_rng(12)
    grid = t[rng.integers(0x30, 0x48, size=(64, 8))] * np.where(rng.random((64, 8)) < .5, -1, 1)
    grid[0, 0] = 448.0                  # pins the block scale to 1
    codes, scales = O.quantize_fp8_blocks(grid, 64)
    assert scales[0] == 1.0
    np.testing.assert_array_equal(O.dequantize_fp8_blocks(codes, scales, 64), grid)


def test_widen_bf16_matches_library():
    x = torch.randn(1000).to(torch.bfloat16)
    np.testing.assert_array_equal(O.widen_bf16(x.view(torch.int16).numpy().view(np.uint16)),
                                  x.to(torch.float64).numpy())


def test_selection_margin_hand_cases():
    """The diagnostic relative gap between the k-th and (k+1)-th largest
    score of each row, worked by hand: row [3, 1, 2, 0.5] at k = 2 has gap
    2 - 1 over 2 = 0.5; row [5, 4.5, 4, 0] has 0.5 / 4.5; the minimum is
    the second.  Exact ties give 0, negative scores divide by |s_k|, and
    keeping every block leaves no gap (inf)."""
    s = np.array([[3.0, 1.0, 2.0, 0.5], [5.0, 4.5, 4.0, 0.0]])
    assert O.selection_margin(s, 2) == pytest.approx(0.5 / 4.5, rel=1e-15)
    assert O.selection_margin(s, 1) == pytest.approx(0.1, rel=1e-15)     # (5 - 4.5) / 5
    assert O.selection_margin(np.array([[2.0, 1.0, 2.0]]), 1) == 0.0
    assert O.selection_margin(np.array([[-1.0, -3.0, -2.0]]), 1) == 1.0
    assert O.selection_margin(s, 4) == float("inf")

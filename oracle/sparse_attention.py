"""fp64 CPU oracle of block-sparse attention with top-k block selection.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) may import, call or link this module; only the tests,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` do.
It shares no code, table or constant generator with the GPU path.

What it computes, one (batch, head) slice at a time, in float64:

* Block partition (paper §2 "Block sparsity"): the L x L attention matrix is
  cut into contiguous query blocks I_i and key blocks J_j of ``b`` tokens
  (the last block holds the remainder); sparsity is the fraction of blocks the
  sparse branch does not evaluate.  The paper's operating point is b = 64
  (appendix "Training Details", Stage-1 table: 64x64 sparse blocks).
* Block selection M_phi (paper §2, Eq. comp-sparse, and §4.1): the paper names
  top-k over blockwise scores as one admissible selector without fixing it.
  Reading used here: score s_ij = mean over the block of the unscaled logits
  q_t . k_u, which by bilinearity is (sum_t q_t) . (sum_u k_u) / (n_i n_j);
  each query block keeps the k key blocks with the largest score under the
  total order (score descending, block index ascending), listed ascending.
  Selection runs on the bf16 inputs (§4.3 keeps mask selection in BF16).
* Sparse branch O_s = A_M(Q, K, V) (§2 Eq. comp-sparse, §4.1): exact softmax
  attention of every query of I_i over the union of its selected key blocks,
  normalised over that union only, with logits tau * q_t . k_u.
* FP8 operand quantisation (E4M3, §4.3 names E4M3 for its W8A8 linears; the
  per-64-token-block power-of-two scales applied to attention operands are a
  reading, not the paper's): OCP e4m3fn, round to nearest even.

Every function works on numpy float64 arrays of one head: q, k, v are [N, d].
"""
from __future__ import annotations

import math

import numpy as np

NEG_INF = -np.inf


# --------------------------------------------------------------------------
# bf16 widening (input plumbing: bf16 bit patterns are exact in float64)
# --------------------------------------------------------------------------
def widen_bf16(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64, exactly (bf16 is the top half of
    an IEEE binary32)."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# Block partition (§2 "Block sparsity")
# --------------------------------------------------------------------------
def block_count(n_tokens: int, block: int) -> int:
    """Number of contiguous blocks of ``block`` tokens covering n_tokens."""
    return -(-n_tokens // block)


def block_sizes(n_tokens: int, block: int) -> np.ndarray:
    """True token count of every block; the last one holds the remainder."""
    nb = block_count(n_tokens, block)
    sizes = np.full(nb, block, dtype=np.int64)
    if nb:
        sizes[-1] = n_tokens - (nb - 1) * block
    return sizes


def keep_count(keep_bp: int, n_key_blocks: int) -> int:
    """Blocks kept per query block for a keep ratio given in basis points:
    ceil(keep_bp * nkb / 10000) in integers, clamped to [1, nkb].  Sparsity
    (§2) is then 1 - k / nkb."""
    k = -(-keep_bp * n_key_blocks // 10000)
    return int(min(max(k, 1), n_key_blocks))


# --------------------------------------------------------------------------
# Block selection M_phi (§2 Eq. comp-sparse; §4.1)
# --------------------------------------------------------------------------
def pool_blocks(x: np.ndarray, block: int) -> np.ndarray:
    """Sum of the token vectors of every block (fp64): xhat_i = sum_{t in I_i} x_t."""
    n, d = x.shape
    nb = block_count(n, block)
    out = np.zeros((nb, d), dtype=np.float64)
    for i in range(nb):
        out[i] = x[i * block:min((i + 1) * block, n)].sum(axis=0)
    return out


def block_scores(q: np.ndarray, k: np.ndarray, block: int) -> np.ndarray:
    """s_ij = (qhat_i . khat_j) / (n_i n_j): the mean unscaled logit of block (i, j).
    Every dot product is evaluated with the same reduction order (an
    elementwise product summed along the channel axis), so blocks with equal
    pooled vectors get bit-identical scores and exact ties stay ties."""
    nq = block_sizes(q.shape[0], block).astype(np.float64)
    nk = block_sizes(k.shape[0], block).astype(np.float64)
    qh, kh = pool_blocks(q, block), pool_blocks(k, block)
    dots = np.empty((qh.shape[0], kh.shape[0]))
    for i0 in range(0, qh.shape[0], 32):
        dots[i0:i0 + 32] = (qh[i0:i0 + 32, None, :] * kh[None, :, :]).sum(axis=-1)
    return dots / (nq[:, None] * nk[None, :])


def topk_ascending(row_scores: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest entries under (score desc, index asc), sorted
    ascending.  -0.0 and +0.0 compare equal."""
    j = np.arange(row_scores.shape[0])
    order = np.lexsort((j, -row_scores))  # last key is primary
    return np.sort(order[:k])


def select_row_topk(scores: np.ndarray, k: int) -> np.ndarray:
    """Per-query-block top-k over key blocks -> idx [nqb, k] (int32, ascending)."""
    nqb, nkb = scores.shape
    if not 1 <= k <= nkb:
        raise ValueError("k out of range")
    return np.stack([topk_ascending(scores[i], k) for i in range(nqb)]).astype(np.int32)


def head_pair_budget(keep_bp: int, nqb: int, nkb: int) -> int:
    """Pairs kept per head by the ragged selection: ceil(keep_bp * nqb * nkb
    / 10000) in integers, clamped to [nqb, nqb * nkb] (every query block keeps
    at least its best key block)."""
    total = -(-keep_bp * nqb * nkb // 10000)
    return int(min(max(total, nqb), nqb * nkb))


def select_head_topk(scores: np.ndarray, keep_bp: int = None, kmax: int = None,
                     budget: int = None):
    """Ragged selection over a whole head (a reading for ragged per-query-block
    work; the paper only fixes sparsity as a global block fraction, §2).

    K pairs are kept (``budget``, else head_pair_budget(keep_bp, ...)): first
    every query block's best key block, then the remaining K - nqb pairs by
    (score desc, i asc, j asc) among pairs not yet taken.  With ``kmax`` given
    (the fixed row stride of an index list), a row that would keep more than
    kmax pairs keeps only its kmax best by (score desc, j asc).  Returns
    (idx [nqb, w] padded with -1, cnt [nqb]) where w is kmax if given, else
    the largest cnt."""
    nqb, nkb = scores.shape
    total = budget if budget is not None else head_pair_budget(keep_bp, nqb, nkb)
    assert nqb <= total <= nqb * nkb
    taken = np.zeros((nqb, nkb), dtype=bool)
    for i in range(nqb):
        taken[i, topk_ascending(scores[i], 1)[0]] = True
    flat = scores.reshape(-1)
    ii, jj = np.divmod(np.arange(nqb * nkb), nkb)
    order = np.lexsort((jj, ii, -flat))
    need = total - nqb
    for p in order:
        if need == 0:
            break
        if not taken[ii[p], jj[p]]:
            taken[ii[p], jj[p]] = True
            need -= 1
    if kmax is not None:
        for i in range(nqb):
            sel = np.nonzero(taken[i])[0]
            if sel.size > kmax:
                # the kmax best of the row's kept pairs, (score desc, j asc)
                best = sel[np.lexsort((sel, -scores[i, sel]))[:kmax]]
                taken[i] = False
                taken[i, best] = True
    cnt = taken.sum(axis=1).astype(np.int32)
    width = kmax if kmax is not None else int(cnt.max())
    idx = np.full((nqb, width), -1, dtype=np.int32)
    for i in range(nqb):
        sel = np.nonzero(taken[i])[0]
        idx[i, :sel.size] = sel
    return idx, cnt


# --------------------------------------------------------------------------
# Sparse branch A_M (§2 Eq. comp-sparse, §3 "exact softmax on a retained
# subset of query-key blocks", §4.1)
# --------------------------------------------------------------------------
def attend_query_block(q_rows, k, v, blocks, block: int, tau: float):
    """Exact softmax attention of the query rows ``q_rows`` over the union of
    the key blocks listed in ``blocks``.  Returns (O rows, LSE rows); an empty
    list gives O = 0 and LSE = -inf."""
    nk = k.shape[0]
    if len(blocks) == 0:
        return (np.zeros((q_rows.shape[0], v.shape[1])),
                np.full(q_rows.shape[0], NEG_INF))
    keys = np.concatenate([np.arange(j * block, min((j + 1) * block, nk))
                           for j in blocks])
    z = tau * (q_rows @ k[keys].T)
    m = z.max(axis=1, keepdims=True)
    e = np.exp(z - m)
    s = e.sum(axis=1, keepdims=True)
    return (e / s) @ v[keys], (m + np.log(s))[:, 0]


def sparse_attention(q, k, v, idx, cnt, block: int, tau: float, qblocks=None):
    """O_t = sum_{u in U_i} softmax_u(tau q_t.k_u) v_u with U_i the union of
    the key blocks idx[i, :cnt[i]]; also LSE_t = log sum_{u in U_i} exp(tau q_t.k_u).
    A query block with cnt = 0 gets O = 0 and LSE = -inf.
    Returns (O [N, d] float64, LSE [N] float64).  With ``qblocks`` given, only
    those query blocks are computed and the other rows are left at O = 0,
    LSE = -inf (for checking sampled outputs of large problems)."""
    n, d = q.shape
    nqb = block_count(n, block)
    out = np.zeros((n, v.shape[1]), dtype=np.float64)
    lse = np.full(n, NEG_INF, dtype=np.float64)
    for i in (range(nqb) if qblocks is None else qblocks):
        rows = slice(i * block, min((i + 1) * block, n))
        out[rows], lse[rows] = attend_query_block(
            q[rows], k, v, idx[i, :int(cnt[i])], block, tau)
    return out, lse


# --------------------------------------------------------------------------
# OCP FP8 E4M3 ("e4m3fn"): 1 sign, 4 exponent (bias 7), 3 mantissa bits; no
# infinities; S.1111.111 is NaN; largest finite magnitude 448 (§4.3 names
# E4M3; format from the OCP 8-bit floating point specification).
# --------------------------------------------------------------------------
E4M3_MAX = 448.0


def e4m3_decode(code: int) -> float:
    """Value of one e4m3fn byte."""
    code = int(code) & 0xFF
    sign = -1.0 if code & 0x80 else 1.0
    exp = (code >> 3) & 0xF
    man = code & 0x7
    if exp == 0xF and man == 0x7:
        return math.nan
    if exp == 0:
        return sign * man * 2.0 ** -9          # subnormal: man/8 * 2^(1-7)
    return sign * (1.0 + man / 8.0) * 2.0 ** (exp - 7)


def e4m3_table() -> np.ndarray:
    """All 256 code values (float64; NaN for the two NaN codes)."""
    return np.array([e4m3_decode(c) for c in range(256)], dtype=np.float64)


_POS_VALUES = e4m3_table()[:127]          # codes 0..126: 0 .. 448, increasing


def e4m3_encode(x: np.ndarray) -> np.ndarray:
    """Round float64 values to the nearest e4m3fn code, ties to the even code
    (even mantissa), saturating magnitudes above 448 to +-448; the sign bit is
    kept, so negative values that round to zero give -0 (0x80).  NaN is not
    accepted."""
    x = np.asarray(x, dtype=np.float64)
    if np.isnan(x).any():
        raise ValueError("NaN input")
    a = np.minimum(np.abs(x), E4M3_MAX)
    hi = np.searchsorted(_POS_VALUES, a, side="left")     # first value >= a
    hi = np.minimum(hi, 126)
    lo = np.maximum(hi - 1, 0)
    exact = _POS_VALUES[hi] == a
    d_lo = a - _POS_VALUES[lo]
    d_hi = _POS_VALUES[hi] - a
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(exact, hi, np.where(pick_hi, hi, lo)).astype(np.uint8)
    return np.where(np.signbit(x), code | 0x80, code).astype(np.uint8)


def fp8_scale_exponent(amax: float) -> int:
    """Smallest integer e with amax <= 448 * 2^e, but at least -126 so that the
    scale 2^e is a normal fp32 number (and an E8M0 code); 0 for an all-zero
    block."""
    if amax == 0.0:
        return 0
    frac, ex = math.frexp(amax)            # amax = frac * 2^ex, frac in [0.5, 1)
    # 448 = 0.875 * 2^9, so amax <= 0.875 * 2^(9+e) <=> e >= ex - 9 (+1 if frac > 0.875)
    return max(ex - 9 + (1 if frac > 0.875 else 0), -126)


def quantize_fp8_blocks(x: np.ndarray, block: int = 64):
    """Per block of ``block`` tokens: scale = 2^e with e = fp8_scale_exponent(amax
    over the block's true tokens and all channels); codes = E4M3(x / scale).
    Returns (codes uint8 [N, d], scales float64 [nb])."""
    n, _ = x.shape
    nb = block_count(n, block)
    codes = np.zeros(x.shape, dtype=np.uint8)
    scales = np.zeros(nb, dtype=np.float64)
    for i in range(nb):
        rows = slice(i * block, min((i + 1) * block, n))
        e = fp8_scale_exponent(float(np.abs(x[rows]).max()))
        scales[i] = 2.0 ** e
        codes[rows] = e4m3_encode(x[rows] / scales[i])
    return codes, scales


def dequantize_fp8_blocks(codes: np.ndarray, scales: np.ndarray, block: int = 64) -> np.ndarray:
    """x_hat = decode(code) * scale of the token's block."""
    table = e4m3_table()
    vals = table[codes.astype(np.int64)]
    rowscale = np.repeat(scales, block)[:codes.shape[0]]
    return vals * rowscale[:, None]


# --------------------------------------------------------------------------
# The whole hot path for one head
# --------------------------------------------------------------------------
def select_head(q, k, block: int, keep_bp: int, mode: str = "row"):
    """Selection for one head from its (widened bf16) q and k.
    mode "row": per-query-block top-k (uniform cnt); mode "head": ragged."""
    s = block_scores(q, k, block)
    if mode == "row":
        kk = keep_count(keep_bp, s.shape[1])
        idx = select_row_topk(s, kk)
        return idx, np.full(s.shape[0], kk, dtype=np.int32)
    if mode == "head":
        return select_head_topk(s, keep_bp)
    raise ValueError(mode)


def selection_margin(scores: np.ndarray, k: int) -> float:
    """Smallest relative gap between the k-th and (k+1)-th score over all rows
    (diagnoses near-ties; inf when k == nkb)."""
    if k >= scores.shape[1]:
        return math.inf
    srt = -np.sort(-scores, axis=1)
    gap = srt[:, k - 1] - srt[:, k]
    den = np.maximum(np.abs(srt[:, k - 1]), 1e-300)
    return float((gap / den).min())

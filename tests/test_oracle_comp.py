"""Pins of the oracle's compensation branch (paper §2 Eq. comp-sparse, §4.1)
against facts independent of it: a library logistic function, rotation
identities, a brute-force sum for the low-rank state, RMSNorm invariants,
the gate's closed form and a hand-derived two-token case."""
import math

import numpy as np
import pytest
from scipy.special import expit

import oracle as O
import workloads as W


def test_silu_matches_logistic_and_odd_part():
    x = np.linspace(-40, 40, 2001)
    assert np.allclose(O.silu(x), x * expit(x), rtol=1e-15, atol=1e-300)
    # silu(x) - silu(-x) = x (sigmoid(x) + sigmoid(-x) = 1)
    assert np.allclose(O.silu(x) - O.silu(-x), x, rtol=1e-14, atol=1e-14)
    assert O.silu(np.array([0.0]))[0] == 0.0


def _table(angles):
    ang = np.asarray(angles, np.float64)
    return np.stack([np.cos(ang), np.sin(ang)], axis=-1)


def test_rope_rotation_convention_and_identities():
    rng = np.random.default_rng(1)
    # counter-clockwise: (1, 0) -> (cos t, sin t), (0, 1) -> (-sin t, cos t)
    t = 0.7
    e = O.rope_rotate(np.array([[1.0, 0.0], [0.0, 1.0]]), _table([[t], [t]]))
    assert np.allclose(e, [[math.cos(t), math.sin(t)], [-math.sin(t), math.cos(t)]], atol=1e-15)
    x = rng.standard_normal((5, 8))
    assert np.array_equal(O.rope_rotate(x, _table(np.zeros((5, 4)))), x)   # zero angle
    a1, a2 = rng.uniform(-9, 9, (5, 4)), rng.uniform(-9, 9, (5, 4))
    y = O.rope_rotate(x, _table(a1))
    pair_norm = lambda z: z[:, 0::2] ** 2 + z[:, 1::2] ** 2
    assert np.allclose(pair_norm(y), pair_norm(x), rtol=1e-13)
    # composition: rotating by a1 then a2 equals rotating by a1 + a2
    assert np.allclose(O.rope_rotate(y, _table(a2)), O.rope_rotate(x, _table(a1 + a2)), atol=1e-12)
    # relative position: <R(ai) a, R(aj) b> = <R(ai - aj) a, b> per pair
    b = rng.standard_normal((5, 8))
    lhs = np.sum(O.rope_rotate(x, _table(a1)) * O.rope_rotate(b, _table(a2)), axis=1)
    rhs = np.sum(O.rope_rotate(x, _table(a1 - a2)) * b, axis=1)
    assert np.allclose(lhs, rhs, atol=1e-12)


def test_state_is_the_sum_of_outer_products():
    rng = np.random.default_rng(2)
    n, d, r = 37, 16, 8
    kn, v = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    pk = rng.standard_normal((r, d)) / 4
    rope = _table(rng.uniform(-5, 5, (n, r // 2)))
    c = O.comp_state(kn, v, pk, rope)
    ref = np.zeros((r, d))
    for j in range(n):                       # brute force, one token at a time
        f = np.array([math.fsum(pk[m, c_] * kn[j, c_] for c_ in range(d)) for m in range(r)])
        f = f / (1.0 + np.exp(-f))           # silu
        rot = np.empty(r)
        for m in range(r // 2):
            cs, sn = rope[j, m]
            rot[2 * m] = f[2 * m] * cs - f[2 * m + 1] * sn
            rot[2 * m + 1] = f[2 * m] * sn + f[2 * m + 1] * cs
        ref += np.outer(rot, v[j])
    assert np.allclose(c, ref, rtol=1e-12, atol=1e-12)


def test_rmsnorm_invariants():
    rng = np.random.default_rng(3)
    n, d, r = 9, 16, 8
    qn = rng.standard_normal((n, d))
    pq = rng.standard_normal((r, d)) / 4
    rope = _table(rng.uniform(-5, 5, (n, r // 2)))
    state = rng.standard_normal((r, d))
    out = O.comp_lowrank(qn, pq, rope, state, gamma=None, eps=0.0)
    assert np.allclose(np.mean(out * out, axis=1), 1.0, rtol=1e-13)       # unit RMS
    out7 = O.comp_lowrank(qn, pq, rope, 7.0 * state, gamma=None, eps=0.0)
    assert np.allclose(out7, out, rtol=1e-13)                               # scale invariant
    gamma = rng.standard_normal(d)
    outg = O.comp_lowrank(qn, pq, rope, state, gamma=gamma, eps=0.0)
    assert np.allclose(outg, out * gamma[None, :], rtol=1e-13)


def test_gate_closed_form():
    o_s = np.array([[3.0, 4.0], [0.0, 0.0], [1.0, -1.0]])
    o_lr = np.array([[1.0, 0.0], [5.0, 5.0], [0.5, 0.25]])
    gate = np.array([2.0, 3.0, 0.0])
    out = O.comp_combine(o_s, o_lr, gate)
    assert np.allclose(out[0], [3.0 + 2.0 * math.sqrt(12.5), 4.0], rtol=1e-15)
    assert np.array_equal(out[1], [0.0, 0.0])      # rms(O_s) = 0 keeps the row
    assert np.array_equal(out[2], o_s[2])          # gate 0 is the sparse branch exactly


def test_two_token_hand_case():
    """d = r = 2, P = I, rope angles 0 and pi/2, eps = 0, gamma = 1:
    k~_0 = (silu 1, 0), k~_1 = R(pi/2)(silu 0, silu 2) = (-silu 2, 0),
    C = k~_0 v_0^T + k~_1 v_1^T has one non-zero row c, so for q_0 = (1, 0)
    the low-rank output is c / rms(c) and O_0 = O_s0 + g rms(O_s0) c / rms(c)."""
    s1 = 1.0 / (1.0 + math.exp(-1.0))
    s2 = 2.0 / (1.0 + math.exp(-2.0))
    v0, v1 = np.array([1.0, 2.0]), np.array([3.0, -1.0])
    c = s1 * v0 - s2 * v1
    rope = np.array([[[1.0, 0.0]], [[0.0, 1.0]]])
    eye = np.eye(2)
    kn = np.array([[1.0, 0.0], [0.0, 2.0]])
    state = O.comp_state(kn, np.stack([v0, v1]), eye, rope)
    assert np.allclose(state, [c, [0.0, 0.0]], rtol=1e-15, atol=1e-15)
    qn = np.array([[1.0, 0.0], [0.0, 1.0]])
    olr = O.comp_lowrank(qn, eye, rope, state, eps=0.0)
    rms_c = math.sqrt((c[0] ** 2 + c[1] ** 2) / 2)
    assert np.allclose(olr[0], c / rms_c, rtol=1e-14)
    o_s = np.array([[0.5, -0.25], [1.0, 1.0]])
    out = O.compensated_output(o_s, qn, kn, np.stack([v0, v1]), eye, eye, rope,
                               np.array([0.3, 0.0]), eps=0.0)
    rms_o = math.sqrt((0.25 + 0.0625) / 2)
    assert np.allclose(out[0], o_s[0] + 0.3 * rms_o * c / rms_c, rtol=1e-14)


def test_rope_table_schedule():
    axis, freq = W.rope_pairs_wan(128)
    assert len(axis) == 64
    assert (axis[:22] == 0).all() and (axis[22:43] == 1).all() and (axis[43:] == 2).all()
    assert freq[0] == 1.0 and freq[22] == 1.0 and freq[43] == 1.0
    assert math.isclose(freq[1], 10000.0 ** (-2.0 / 44), rel_tol=1e-15)
    t = W.rope_table((3, 4, 5), 64)
    assert t.shape == (60, 32, 2) and t.dtype == np.float32
    # token (t=2, y=1, x=3) is index (2*4 + 1)*5 + 3 = 48; pair 1 turns with t, pair 23 with y
    assert math.isclose(t[48, 1, 0], math.cos(2 * freq[1]), rel_tol=1e-6)
    assert math.isclose(t[48, 23, 1], math.sin(1 * freq[23]), rel_tol=1e-6)
    assert np.allclose(np.sum(t.astype(np.float64) ** 2, axis=-1), 1.0, atol=1e-6)


# ---- causal window -----------------------------------------------------------
def _causal_case(n=37, d=8, r=4, seed=21):
    rng = np.random.default_rng(seed)
    kn, v, qn = (rng.standard_normal((n, d)) for _ in range(3))
    pk, pq = (rng.standard_normal((r, d)) / math.sqrt(d) for _ in range(2))
    ang = rng.uniform(0, 2 * np.pi, (n, r // 2))
    rope = np.stack([np.cos(ang), np.sin(ang)], axis=-1)
    return qn, kn, v, pq, pk, rope


@pytest.mark.parametrize("chunk,window", [(10, 0), (10, 1), (8, 2), (37, 0), (5, 3)])
def test_causal_state_is_the_sum_over_each_querys_allowed_keys(chunk, window):
    """Per token t, brute force over the pairs (t, j) with j in chunks
    [c(t) - W + 1, c(t)]: the outer products summed one by one with fsum
    equal the state the oracle keeps for t's chunk."""
    qn, kn, v, pq, pk, rope = _causal_case()
    n = kn.shape[0]
    states = O.comp_state_causal(kn, v, pk, rope, chunk, window)
    kt = O.comp_features(kn, pk, rope)
    for t in (0, 9, 10, 19, 23, 36):
        ct = t // chunk
        keys = [j for j in range(n)
                if j // chunk <= ct and (window == 0 or j // chunk > ct - window)]
        ref = np.array([[math.fsum(kt[j, m] * v[j, c] for j in keys) for c in range(v.shape[1])]
                        for m in range(kt.shape[1])])
        assert np.allclose(states[ct], ref, rtol=1e-12, atol=1e-12), (t, chunk, window)


def test_causal_one_chunk_is_the_unrestricted_branch():
    qn, kn, v, pq, pk, rope = _causal_case(seed=22)
    rng = np.random.default_rng(23)
    o_s = rng.standard_normal(qn.shape)
    gate = rng.standard_normal(qn.shape[0])
    a = O.compensated_output_causal(o_s, qn, kn, v, pq, pk, rope, gate, qn.shape[0], 0)
    b = O.compensated_output(o_s, qn, kn, v, pq, pk, rope, gate)
    assert np.allclose(a, b, rtol=1e-13, atol=1e-13)


def test_causal_window_one_is_block_diagonal():
    """Window 1: each chunk's state is the unrestricted state of that chunk's
    tokens alone, and the output of a chunk does not change when the other
    chunks' keys and values change."""
    qn, kn, v, pq, pk, rope = _causal_case(seed=24)
    chunk = 10
    states = O.comp_state_causal(kn, v, pk, rope, chunk, 1)
    for c in range(states.shape[0]):
        sl = slice(c * chunk, (c + 1) * chunk)
        assert np.allclose(states[c], O.comp_state(kn[sl], v[sl], pk, rope[sl]),
                           rtol=1e-13, atol=1e-13)
    rng = np.random.default_rng(25)
    o_s = rng.standard_normal(qn.shape)
    gate = rng.standard_normal(qn.shape[0])
    a = O.compensated_output_causal(o_s, qn, kn, v, pq, pk, rope, gate, chunk, 1)
    kn2, v2 = kn.copy(), v.copy()
    kn2[:10] += 1.0
    v2[20:] -= 2.0
    b = O.compensated_output_causal(o_s, qn, kn2, v2, pq, pk, rope, gate, chunk, 1)
    assert np.array_equal(a[10:20], b[10:20])

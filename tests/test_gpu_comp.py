"""GPU parity of the compensation branch and gate epilogue (paper §2 Eq.
comp-sparse, §4.1) through the C ABI against the fp64 oracle on identical
seeded inputs: the low-rank state and the gated output within the bf16 bar,
a zero gate returning O_s bit-exactly.

The gated output is O_s plus g * rms(O_s) * O_lr with O_lr of unit RMS, so
its entries reach several units, where one bf16 rounding alone is up to
|O| * 2^-9; the element bar is therefore 2e-2 * max(1, |O_ref|) (the bf16 bar
of the attention output, scaled by the output's magnitude above one), and
the rel-L2 bar stays 1e-2."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2609_23153_amd as sa
import workloads as W
from gpu_helpers import rel_l2, say, widen

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
R = sa.COMP_RANK


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sa.library()
    yield
    torch.cuda.synchronize()


def inputs(grid, heads=2, batch=1, seed=0, gen="locality"):
    wl = W.Workload("comp", batch, heads, grid, 128, 64, 1000, gen, seed)
    qn, kn, v = W.make_inputs(wl)
    g = torch.Generator().manual_seed(seed + 77)
    o_s = torch.randn(qn.shape, generator=g).to(torch.bfloat16)
    pq, pk, gamma, gate = W.comp_params(wl, R, seed_extra=seed)
    rope = torch.from_numpy(W.rope_table(grid, R))
    return wl, qn, kn, v, o_s, pq, pk, gamma, gate, rope


def run_gpu(qn, kn, v, o_s, pq, pk, gamma, gate, rope, eps=1e-6, inplace=False):
    d = lambda t: None if t is None else t.to(DEV)
    qd, kd, vd, od, pqd, pkd, gd, gtd, rd = map(d, (qn, kn, v, o_s, pq, pk, gamma, gate, rope))
    state = sa.sparse_attn_comp_state(kd, vd, pkd, rd)
    out = od if inplace else None
    o = sa.sparse_attn_comp_out(qd, pqd, rd, state, gtd, od, gamma=gd, eps=eps, o=out)
    torch.cuda.synchronize()
    return state.cpu().numpy(), o.cpu()


def check_head(b, h, qn, kn, v, o_s, pq, pk, gamma, gate, rope, state, o, what, eps=1e-6,
               rows=None):
    rp = rope.numpy()
    ref_state = O.comp_state(widen(kn[b, h]), widen(v[b, h]), widen(pk[h]), rp)
    es = rel_l2(state[b, h].T, ref_state)          # the state is stored as C^T
    g = None if gamma is None else gamma[h].double().numpy()
    olr = O.comp_lowrank(widen(qn[b, h]), widen(pq[h]), rp, ref_state, g, eps)
    ref = O.comp_combine(widen(o_s[b, h]), olr, gate[b, h].double().numpy())
    got = o[b, h].to(torch.float64).numpy()
    if rows is not None:
        got, ref = got[rows], ref[rows]
    eo = rel_l2(got, ref)
    scaled = float((np.abs(got - ref) / np.maximum(1.0, np.abs(ref))).max())
    say(f"  {what} b{b} h{h}: state rel_l2={es:.3e}  out rel_l2={eo:.3e} "
        f"max |err|/max(1,|ref|)={scaled:.3e}")
    assert es <= 1e-2, (what, es)
    assert eo <= 1e-2 and scaled <= 2e-2, (what, eo, scaled)


@pytest.mark.parametrize("grid", [(4, 16, 32), (5, 8, 25), (3, 7, 11)])
def test_comp_small(grid):
    """Token counts 2048 (one chunk), 1000 and 231 (ragged sub-tiles)."""
    _, qn, kn, v, o_s, pq, pk, gamma, gate, rope = inputs(grid, heads=2, batch=2, seed=1)
    state, o = run_gpu(qn, kn, v, o_s, pq, pk, gamma, gate, rope)
    for b in range(2):
        for h in range(2):
            check_head(b, h, qn, kn, v, o_s, pq, pk, gamma, gate, rope, state, o, f"grid {grid}")


def test_comp_multi_chunk_inplace_broadcast_gate_no_gamma():
    """5000 tokens (3 state chunks), output written over O_s, one gate per
    token shared by the heads (head stride 0), RMSNorm without weight."""
    _, qn, kn, v, o_s, pq, pk, _, gate, rope = inputs((5, 40, 25), heads=3, seed=2, gen="normal")
    shared = gate[:, :1, :].to(DEV).expand(-1, 3, -1)  # stride 0 over heads, on the device
    assert shared.stride(1) == 0
    state, o = run_gpu(qn, kn, v, o_s.clone(), pq, pk, None, shared, rope, inplace=True)
    shared = shared.cpu().contiguous()
    for h in range(3):
        check_head(0, h, qn, kn, v, o_s, pq, pk, None, shared, rope, state, o,
                   "in place, shared gate")


def test_comp_zero_gate_is_sparse_branch_exactly():
    _, qn, kn, v, o_s, pq, pk, gamma, gate, rope = inputs((2, 8, 16), seed=3)
    state, o = run_gpu(qn, kn, v, o_s, pq, pk, gamma, torch.zeros_like(gate), rope)
    assert torch.equal(o.view(torch.int16), o_s.view(torch.int16))


def test_comp_full_size_heads():
    """The 14B-720P layer shape (L = 75600, 37 state chunks, a ragged last
    sub-tile): two heads of the 40, all tokens."""
    grid = (21, 45, 80)
    wl = W.Workload("comp_full", 1, 40, grid, 128, 64, 300, "positional", 2)
    heads = [0, 39]
    qn, kn, v = W.make_inputs(wl, heads=heads)
    g = torch.Generator().manual_seed(5)
    o_s = torch.randn(qn.shape, generator=g).to(torch.bfloat16)
    pq, pk, gamma, gate = W.comp_params(wl, R)
    pq, pk, gamma = pq[heads].contiguous(), pk[heads].contiguous(), gamma[heads].contiguous()
    gate = gate[:, heads].contiguous()
    rope = torch.from_numpy(W.rope_table(grid, R))
    state, o = run_gpu(qn, kn, v, o_s, pq, pk, gamma, gate, rope)
    for i in range(len(heads)):
        check_head(0, i, qn, kn, v, o_s, pq, pk, gamma, gate, rope, state, o, "14B-720P")


# ---- causal window -----------------------------------------------------------
def check_head_causal(b, h, qn, kn, v, o_s, pq, pk, gamma, gate, rope, state, o, causal, what,
                      rows=None):
    """State per chunk and gated output against the oracle's causal branch."""
    rp = rope.numpy()
    chunk, window = causal
    ref_states = O.comp_state_causal(widen(kn[b, h]), widen(v[b, h]), widen(pk[h]), rp, chunk,
                                     window)
    assert state.shape[2] == ref_states.shape[0], (what, state.shape)
    es = max(rel_l2(state[b, h, c].T, ref_states[c]) for c in range(ref_states.shape[0]))
    g = None if gamma is None else gamma[h].double().numpy()
    olr = O.comp_lowrank_causal(widen(qn[b, h]), widen(pq[h]), rp, ref_states, chunk, g, 1e-6)
    ref = O.comp_combine(widen(o_s[b, h]), olr, gate[b, h].double().numpy())
    got = o[b, h].to(torch.float64).numpy()
    if rows is not None:
        got, ref = got[rows], ref[rows]
    eo = rel_l2(got, ref)
    scaled = float((np.abs(got - ref) / np.maximum(1.0, np.abs(ref))).max())
    say(f"  {what} b{b} h{h}: {ref_states.shape[0]} states, worst rel_l2={es:.3e}  out "
        f"rel_l2={eo:.3e} max |err|/max(1,|ref|)={scaled:.3e}")
    assert es <= 1e-2, (what, es)
    assert eo <= 1e-2 and scaled <= 2e-2, (what, eo, scaled)


def run_gpu_causal(qn, kn, v, o_s, pq, pk, gamma, gate, rope, causal):
    d = lambda t: None if t is None else t.to(DEV)
    qd, kd, vd, od, pqd, pkd, gd, gtd, rd = map(d, (qn, kn, v, o_s, pq, pk, gamma, gate, rope))
    state = sa.sparse_attn_comp_state(kd, vd, pkd, rd, causal=causal)
    o = sa.sparse_attn_comp_out(qd, pqd, rd, state, gtd, od, gamma=gd, causal=causal)
    torch.cuda.synchronize()
    return state.cpu().numpy(), o.cpu()


@pytest.mark.parametrize("grid,causal", [((4, 16, 32), (1024, 0)), ((4, 16, 32), (1024, 2)),
                                         ((4, 16, 32), (2048, 1)), ((5, 8, 25), (300, 0)),
                                         ((3, 7, 11), (77, 2)), ((6, 20, 25), (1500, 0))])
def test_comp_causal(grid, causal):
    """Chunks of whole frames and chunk boundaries inside 128-token tiles and
    1024-token sub-chunks (300, 77, 1500 tokens), windows 0, 1, 2."""
    wl, qn, kn, v, o_s, pq, pk, gamma, gate, rope = inputs(grid, seed=sum(grid) + causal[0])
    state, o = run_gpu_causal(qn, kn, v, o_s, pq, pk, gamma, gate, rope, causal)
    for h in range(qn.shape[1]):
        check_head_causal(0, h, qn, kn, v, o_s, pq, pk, gamma, gate, rope, state, o, causal,
                          f"causal {grid} {causal}")


def test_comp_causal_one_chunk_equals_unrestricted():
    """A single chunk covering the sequence: state and output equal the
    unrestricted calls bit for bit."""
    wl, qn, kn, v, o_s, pq, pk, gamma, gate, rope = inputs((4, 16, 32), seed=9)
    s0, o0 = run_gpu(qn, kn, v, o_s, pq, pk, gamma, gate, rope)
    s1, o1 = run_gpu_causal(qn, kn, v, o_s, pq, pk, gamma, gate, rope, (qn.shape[2], 0))
    assert np.array_equal(s0, s1[:, :, 0])
    assert torch.equal(o0.view(torch.int16), o1.view(torch.int16))


def test_comp_causal_full_size_heads():
    """The 14B-720P shape generated in chunks of 3 latent frames (10,800
    tokens, full history: 7 states per head): two heads whole."""
    grid = (21, 45, 80)
    wl, qn, kn, v, o_s, pq, pk, gamma, gate, rope = inputs(grid, heads=2, seed=31)
    causal = (3 * 45 * 80, 0)
    state, o = run_gpu_causal(qn, kn, v, o_s, pq, pk, gamma, gate, rope, causal)
    for h in range(2):
        check_head_causal(0, h, qn, kn, v, o_s, pq, pk, gamma, gate, rope, state, o, causal,
                          "14B-720P causal")

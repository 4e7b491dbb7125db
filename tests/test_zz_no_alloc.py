"""The allocation-free schedule entry point (sparse_attn_schedule_static),
through the C ABI, against sparse_attn_schedule with a caller workspace:
the same launch order bit for bit, on two calls in a row, the second on a
smaller problem (the per-GPU device array keeps the first call's counters,
which the second must not depend on)."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2609_23153_amd as sa
from gpu_helpers import check_launch_order, say

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def desc_for(B, H, N, block):
    d = sa.SparseAttnDesc()
    d.batch, d.heads, d.seqlen, d.head_dim, d.block = B, H, N, 128, block
    return d


def run_both(cnt_np, N, kmax, block):
    B, H, _ = cnt_np.shape
    cnt = torch.from_numpy(cnt_np).to(DEV)
    lib = sa.library()
    d = desc_for(B, H, N, block)
    G = lib.sparse_attn_num_tiles(ctypes.byref(d))
    ref = torch.full((G,), -7, dtype=torch.int32, device=DEV)
    ws = torch.empty(lib.sparse_attn_workspace_size(ctypes.byref(d), sa.SA_OP_SCHEDULE, kmax),
                     dtype=torch.uint8, device=DEV)
    st = lib.sparse_attn_schedule(ctypes.byref(d), cnt.data_ptr(), kmax, ref.data_ptr(),
                                  ws.data_ptr(), ws.numel(), None)
    assert st == 0
    got = torch.full((G,), -9, dtype=torch.int32, device=DEV)
    st = lib.sparse_attn_schedule_static(ctypes.byref(d), cnt.data_ptr(), kmax, got.data_ptr(),
                                         None)
    assert st == 0
    torch.cuda.synchronize()
    return ref.cpu().numpy(), got.cpu().numpy()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    sa.library()
    yield
    torch.cuda.synchronize()


def test_schedule_static_matches_workspace_entry_point():
    rng = np.random.default_rng(31)
    # first call: 3 x 40 heads of 1182 ragged lists (139 chunks of 1024 tiles)
    big = rng.integers(0, 300, size=(3, 40, 1182)).astype(np.int32)
    big[0, 0, :50] = 0
    ref, got = run_both(big, 75600, 250, 64)
    assert np.array_equal(ref, got)
    check_launch_order(got, big, 250, 75600, 64, "static, large")
    say(f"  static schedule, {ref.size} tiles: identical")
    # second call, smaller: 1 x 12 heads at block 128 (7 chunks); the array
    # still holds the larger call's counters
    small = rng.integers(0, 40, size=(1, 12, 256)).astype(np.int32)
    ref, got = run_both(small, 32760, 40, 128)
    assert np.array_equal(ref, got)
    check_launch_order(got, small, 40, 32760, 128, "static, small")
    say(f"  static schedule, {ref.size} tiles: identical")
    # the binding wrapper on the 14B-720P shape's uniform lists
    cnt = torch.full((1, 40, 1182), 36, dtype=torch.int32, device=DEV)
    order = torch.empty(40 * 1182, dtype=torch.int32, device=DEV)
    sa.sparse_attn_schedule_static(cnt, 75600, 36, order)
    ref = sa.sparse_attn_schedule(cnt, 75600, 36)
    torch.cuda.synchronize()
    assert torch.equal(order, ref)

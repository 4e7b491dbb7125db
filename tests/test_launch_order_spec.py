"""CPU checks of the launch-order property checker that the GPU tests apply
to sparse_attn_schedule: it accepts the orders the header's definition gives
on hand-worked cases and rejects orders that break a property (so a GPU test
passing through it is not vacuous).  The order is this library's own choice;
the paper fixes none."""
import numpy as np
import pytest

from gpu_helpers import check_launch_order, sorted_position, tile_classes


def test_sorted_position_is_a_bijection():
    for G in (1, 7, 2048, 2049, 5000, 3 * 2048):
        pos = [sorted_position(s, G) for s in range(G)]
        assert sorted(pos) == list(range(G))


def test_hand_worked_orders():
    # fewer tiles than one XCD group of 2048: sorted order itself
    cnt = np.full((1, 2, 10), 3)
    check_launch_order(np.arange(20), cnt, 3, 640, 64)
    # ragged: classes of costs 1, 4, 0, 2 are 1, 3, 0, 2 -> tiles 1, 3, 0, 2
    cnt = np.array([[[1, 4, 0, 2]]])
    assert tile_classes(cnt, 9, 256, 64).tolist() == [1, 3, 0, 2]
    check_launch_order([1, 3, 0, 2], cnt, 9, 256, 64)
    # block 128: one list per two 64-row tiles, cost doubled, cnt clamped to kmax
    cnt = np.array([[[5, 1]]])
    assert tile_classes(cnt, 2, 256, 128).tolist() == [3, 3, 2, 2]
    check_launch_order([0, 1, 2, 3], cnt, 2, 256, 128)
    # one full group of 8 x 256 uniform tiles: slot s goes to XCD s % 8,
    # which walks its own run of 256 consecutive tiles
    cnt = np.full((1, 1, 2048), 1)
    o = np.empty(2048, dtype=np.int64)
    for s in range(2048):
        o[s] = 256 * (s % 8) + s // 8
    assert o[:9].tolist() == [0, 256, 512, 768, 1024, 1280, 1536, 1792, 1]
    check_launch_order(o, cnt, 1, 2048 * 64, 64)


def test_checker_rejects_broken_orders():
    cnt = np.array([[[1, 4, 0, 2]]])
    with pytest.raises(AssertionError):
        check_launch_order([1, 3, 2, 0], cnt, 9, 256, 64)   # classes increase
    with pytest.raises(AssertionError):
        check_launch_order([1, 3, 0, 0], cnt, 9, 256, 64)   # not a permutation
    cnt = np.full((1, 2, 10), 3)
    with pytest.raises(AssertionError):
        check_launch_order([1, 0] + list(range(2, 20)), cnt, 3, 640, 64)  # ties out of order
    cnt = np.full((1, 1, 2048), 1)
    with pytest.raises(AssertionError):
        check_launch_order(np.arange(2048), cnt, 1, 2048 * 64, 64)  # no XCD interleave

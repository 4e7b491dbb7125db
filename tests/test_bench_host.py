"""Host logic of bench.py that its reported numbers rest on: the algorithmic
flops of the fused forward over the selected block pairs (the roofline's
`achieved` numerator), checked against a brute-force count over ragged lists,
and the HBM traffic figure, which must follow the committed counter summary
only while the kernel sources it was taken on are unchanged."""
import hashlib
import os

import numpy as np

import bench


def brute_flops(cnt, idx, N, block, d):
    B, H, nb = cnt.shape
    kmax = idx.shape[-1]
    total = 0
    for b in range(B):
        for h in range(H):
            for i in range(nb):
                ni = min(block, N - i * block)
                for p in range(min(max(int(cnt[b, h, i]), 0), kmax)):
                    j = int(idx[b, h, i, p])
                    if 0 <= j < nb:
                        total += 4 * d * ni * min(block, N - j * block)
    return total


def test_selected_flops_matches_pair_count():
    rng = np.random.default_rng(3)
    for N, block in [(1000, 64), (777, 128), (64 * 9, 64)]:
        nb = -(-N // block)
        B, H, kmax = 2, 3, 6
        idx = rng.integers(-1, nb + 2, size=(B, H, nb, kmax)).astype(np.int32)  # -1 and >= nb skipped
        cnt = rng.integers(-1, kmax + 2, size=(B, H, nb)).astype(np.int32)      # clamped to [0, kmax]
        cnt[0, 0, 0], cnt[0, 0, 1] = 0, kmax
        assert bench.selected_flops(cnt, idx, N, block, 128) == brute_flops(cnt, idx, N, block, 128)


def test_selected_flops_dense_lists_equal_dense_attention():
    N, block, d = 1000, 64, 128
    nb = -(-N // block)
    idx = np.tile(np.arange(nb, dtype=np.int32), (1, 2, nb, 1))
    cnt = np.full((1, 2, nb), nb, dtype=np.int32)
    assert bench.selected_flops(cnt, idx, N, block, d) == 2 * 4 * N * N * d


def test_traffic_follows_the_summary_only_while_sources_match(tmp_path, monkeypatch):
    """Per-kernel counter traffic is reported for the summarised workload,
    and only while the kernel's sources hash to the recorded value."""
    prof = tmp_path / "traffic.txt"
    lines = ["# synthetic summary"]
    for i, kern in enumerate(bench.TRAFFIC_SOURCES):
        lines += [f"{kern}.workload: wan14b_720p", f"{kern}.source_sha256: {bench.source_hash(kern)}",
                  f"{kern}.traffic_bytes_per_launch: {1000 + i}"]
    prof.write_text("\n".join(lines) + "\n")
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(prof))
    for i, kern in enumerate(bench.TRAFFIC_SOURCES):
        assert bench.measured_traffic(kern, "wan14b_720p") == 1000 + i
        assert bench.measured_traffic(kern, "wan13b_480p") is None  # other workload
    assert bench.sel_traffic("wan14b_720p") == (1000 + list(bench.TRAFFIC_SOURCES).index("pool_kernel")
                                              + 1000 + list(bench.TRAFFIC_SOURCES).index("score_topk_kernel"))
    stale = prof.read_text().replace(bench.source_hash("fwd_fp8_kernel"), "0" * 64)
    prof.write_text(stale)
    assert bench.measured_traffic("fwd_fp8_kernel", "wan14b_720p") is None
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(tmp_path / "missing.txt"))
    assert bench.measured_traffic("fwd_bf16_kernel", "wan14b_720p") is None

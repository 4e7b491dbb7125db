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


def _summary_values():
    kv = {}
    for line in open(bench.TRAFFIC_PROFILE):
        if not line.startswith("#") and ":" in line:
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    return kv


def _source_hash():
    h = hashlib.sha256()
    for f in bench.FWD_BF16_SOURCES:
        with open(os.path.join(bench.ROOT, "paper_2609_23153_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def test_traffic_follows_the_committed_summary_only_while_sources_match(tmp_path, monkeypatch):
    kv = _summary_values()
    expect = int(float(kv["traffic_bytes_per_launch"]))
    got = bench.measured_traffic("wan14b_720p")
    assert got == (expect if kv["fwd_bf16_source_sha256"] == _source_hash() else None)
    assert bench.measured_traffic("wan13b_480p") is None  # counters cover one workload only
    stale = tmp_path / "traffic.txt"
    stale.write_text(open(bench.TRAFFIC_PROFILE).read().replace(
        kv["fwd_bf16_source_sha256"], "0" * 64))
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(stale))
    assert bench.measured_traffic("wan14b_720p") is None

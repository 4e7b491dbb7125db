#!/usr/bin/env python3
"""Benchmark of the block-sparse attention hot path on one MI355X.

A step is one pass of the whole path over one layer's synthetic inputs, all
resident in HBM before timing starts: block selection (pool + fp64 score +
top-k), work scheduling, and the fused sparse forward, all in the HIP library.
Default workload: the Wan2.1-T2V-14B 720P attention layer shape (B=1, H=40,
L=75,600 tokens = 21x45x80 latent grid, d=128) at 97% block sparsity
(64x64 blocks, 36 of 1182 key blocks kept per query block), bf16.

Prints one JSON line.  `value` is the dense-equivalent TFLOP/s of the whole
step (4*B*H*L^2*d flops of the dense attention the step replaces, divided by
the step time); `roofline` reports the fused forward kernel's actual flops
over the selected blocks against the bf16 MFMA peak, timed with HIP events on
the stream the kernels run on; `cpu_baseline` times the fp64 CPU oracle on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402
import torch  # noqa: E402

METRIC = "ms/call + dense-equiv TFLOP/s and % MFMA peak, block-sparse attn @97%"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0    # MI355X dense fp8 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "hbm_traffic_wan14b_720p.txt")
# sources each kernel's counters depend on (sched.hip: the launch order;
# quant_fp8.hip: the fp8 operand layout)
TRAFFIC_SOURCES = {
    "fwd_bf16_kernel": ("fwd_bf16.hip", "common.h", "launch.h", "sched.hip"),
    "fwd_fp8_kernel": ("fwd_fp8.hip", "quant_fp8.hip", "common.h", "launch.h", "sched.hip"),
    "pool_kernel": ("select.hip", "common.h", "launch.h"),
    "score_topk_kernel": ("select.hip", "common.h", "launch.h"),
}


def source_hash(kernel):
    h = hashlib.sha256()
    for f in TRAFFIC_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2609_23153_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (copy-calibrated), or None when that
    summary does not cover the kernel on this workload or the kernel's sources
    have changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_PROFILE):
        return None
    kv = {}
    for line in open(TRAFFIC_PROFILE):
        if not line.startswith("#") and ":" in line:
            key, val = line.split(":", 1)
            kv[key.strip()] = val.strip()
    if kv.get(f"{kernel}.workload") != workload:
        return None
    if kv.get(f"{kernel}.source_sha256") != source_hash(kernel):
        return None
    return int(float(kv[f"{kernel}.traffic_bytes_per_launch"]))


def sel_traffic(workload):
    """HBM bytes of the selection call (pool + on-chip score/top-k), when both
    kernels' counters cover the workload and sources."""
    a, b = measured_traffic("pool_kernel", workload), measured_traffic("score_topk_kernel", workload)
    return None if a is None or b is None else a + b


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="wan14b_720p")
    ap.add_argument("--cpu-baseline", choices=["on", "off"], default="on")
    ap.add_argument("--cpu-heads", type=int, default=16,
                    help="heads of the workload the oracle runs for the CPU baseline (spread "
                         "evenly over the layer; the time is scaled to all heads)")
    ap.add_argument("--wan13b", choices=["on", "off"], default="on",
                    help="also time select + schedule + fwd on the Wan2.1-1.3B 480P layer")
    ap.add_argument("--normal", choices=["on", "off"], default="on",
                    help="also time select + schedule + fwd at the 14B-720P shape on i.i.d. "
                         "normal inputs (lists without locality)")
    ap.add_argument("--cold", choices=["on", "off"], default="on",
                    help="also time every call with the caches flushed before it (a 512 MB "
                         "scratch overwrite)")
    ap.add_argument("--fp8", choices=["on", "off"], default="on",
                    help="also time the fp8 path on the outlier workload of the same shape")
    ap.add_argument("--comp", choices=["on", "off"], default="on",
                    help="also time the compensation branch and gate epilogue on the bf16 "
                         "layer's inputs and sparse output")
    ap.add_argument("--linear", choices=["on", "off"], default="on",
                    help="also time the W8A8 fp8 linear layer (per-token quantisation + "
                         "fp8 GEMM) at the 14B-720P q/k/v/o projection shape")
    ap.add_argument("--causal", choices=["on", "off"], default="on",
                    help="also time the causal-window variant (auto-regressive generation in "
                         "chunks of 3 latent frames, full history) on the same layer")
    ap.add_argument("--bwd", choices=["on", "off"], default="on",
                    help="also time the backward of the sparse branch (dQ, dK, dV) on the "
                         "bf16 layer's inputs, output and LSE with a synthetic upstream dO")
    ap.add_argument("--sweep", choices=["on", "off"], default="on",
                    help="also time select + schedule + fwd over the sparsity sweep (blocks 64 "
                         "and 128 x keep 3/10/25/100%%) on the locality inputs at the 14B-720P "
                         "shape")
    ap.add_argument("--copy-calib", action="store_true",
                    help="also time a plain 1 GiB device copy (HBM counter calibration)")
    return ap.parse_args()


def selected_flops(cnt, idx, N, block, d):
    """Algorithmic flops of the fused forward: 4 * n_i * n_j * d over every
    selected (query block i, key block j) pair (QK^T and PV, 2 flops/MAC)."""
    nb = cnt.shape[-1]
    sizes = np.full(nb, block, dtype=np.int64)
    sizes[-1] = N - (nb - 1) * block
    kmax = idx.shape[-1]
    valid = np.arange(kmax)[None, None, None, :] < cnt[..., None]
    ok = valid & (idx >= 0) & (idx < nb)  # entries the kernels skip add nothing
    nj = np.where(ok, sizes[np.clip(idx, 0, nb - 1)], 0).sum(-1)  # [B,H,nb]
    return int(4 * d * (nj * sizes[None, None, :]).sum())


def blas_threads():
    """Threads of the BLAS that NumPy (the oracle) runs on."""
    try:
        from threadpoolctl import threadpool_info
        n = [p["num_threads"] for p in threadpool_info() if p.get("user_api") == "blas"]
        if n:
            return int(max(n))
    except Exception:
        pass
    return len(os.sched_getaffinity(0))


def log(msg):
    """Progress line on stderr (stdout carries only the JSON line)."""
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def cpu_model():
    """Model name of the host CPU (from /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


SCRATCH_BYTES = 512 << 20


class CacheFlush:
    """Overwrites a 512 MB device buffer: more than the MI355X's 256 MB
    Infinity Cache plus its 8 x 4 MB of L2, so the call after it starts with
    cold caches (inputs resident in HBM only)."""

    def __init__(self, dev):
        self.buf = torch.empty(SCRATCH_BYTES // 4, dtype=torch.int32, device=dev)
        self.n = 0

    def __call__(self):
        self.n += 1
        self.buf.fill_(self.n)


def time_calls(phases, steps, warmup, flush=None):
    """Per-phase HIP-event times (ms) of `steps` repetitions of the phases
    [(name, fn), ...], after `warmup` untimed repetitions, all on the current
    stream (the stream the library launches on).  Warm: the phases run back
    to back.  Cold (flush given): the cache flush runs before every timed
    phase, outside its events.  Returns {name: [ms, ...]}."""
    for _ in range(warmup):
        for _, fn in phases:
            fn()
    torch.cuda.synchronize()
    ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in phases] for _ in range(steps)]
    for s_ in range(steps):
        for (_, fn), (e0, e1) in zip(phases, ev[s_]):
            if flush is not None:
                flush()
            e0.record()
            fn()
            e1.record()
    torch.cuda.synchronize()
    return {name: [ev[s_][i][0].elapsed_time(ev[s_][i][1]) for s_ in range(steps)]
            for i, (name, _) in enumerate(phases)}


def med(x):
    return round(float(np.median(x)), 4)


def bench_comp(args, sa, W, dev, wl, q, k, v, o_s, sparse_ms):
    """Compensation branch and gate epilogue at the same shape: the low-rank
    state from K and V, then the gated output from Q and the sparse branch's
    output (the layer's Q and K stand in for the normalised queries and keys;
    rank-64 projections, RMSNorm weights and gates are synthetic)."""
    B, H, N, d = q.shape
    r = sa.COMP_RANK
    pq, pk, gamma, gate = (t.to(dev) for t in W.comp_params(wl, r))
    rope = torch.from_numpy(W.rope_table(wl.grid, r)).to(dev)
    state = torch.empty(B, H, d, r, dtype=torch.float32, device=dev)
    desc = sa.make_desc(k, k, v)
    ws = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_COMP_STATE, 1),
                     dtype=torch.uint8, device=dev)
    o = torch.empty_like(o_s)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]

    def step(e=None):
        if e:
            e[0].record()
        sa.sparse_attn_comp_state(k, v, pk, rope, state=state, ws=ws)
        if e:
            e[1].record()
        sa.sparse_attn_comp_out(q, pq, rope, state, gate, o_s, gamma=gamma, o=o)
        if e:
            e[2].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for s_ in range(args.steps):
        step(ev[s_])
    torch.cuda.synchronize()
    st_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    out_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    tok = B * H * N
    rope_b = N * (r // 2) * 2 * 4
    st_bytes = 2 * tok * d * 2 + rope_b + H * r * d * 2 + B * H * r * d * 4
    out_bytes = 3 * tok * d * 2 + rope_b + H * r * d * 2 + B * H * r * d * 4 + tok * 4 + H * d * 4
    gbs = lambda b_, ms: b_ / (ms * 1e-3) / 1e9
    return {
        "ms_per_call": {"comp_state": round(st_ms, 4), "comp_out": round(out_ms, 4)},
        "compensated_step_ms": round(sparse_ms + st_ms + out_ms, 4),
        "rank": r,
        "roofline": {
            "kernels": ["comp_state_kernel", "comp_out_kernel"], "bound": "hbm",
            "achieved": round(gbs(st_bytes + out_bytes, st_ms + out_ms), 1),
            "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(gbs(st_bytes + out_bytes, st_ms + out_ms) / PEAK_HBM_GBS, 4),
            "traffic": None, "algorithmic_bytes": {"comp_state": st_bytes, "comp_out": out_bytes},
        },
        "gbs": {"comp_state": round(gbs(st_bytes, st_ms), 1),
                "comp_out": round(gbs(out_bytes, out_ms), 1)},
    }


def bench_causal(args, sa, W, dev, wl, q, k, v):
    """The sparse branch restricted to a causal window: the same layer
    generated auto-regressively in chunks of 3 latent frames (3 x 45 x 80 =
    10,800 tokens), every earlier chunk visible.  Selection ranks only the
    candidate key blocks (k = 36 of them where there are that many); the
    forward masks keys outside each query's window."""
    B, H, N, d, block = wl.batch, wl.heads, wl.seqlen, wl.head_dim, wl.block
    nb = -(-N // block)
    k_keep = sa.sparse_attn_keep_count(wl.keep_bp, nb)
    chunk = 3 * wl.grid[1] * wl.grid[2]
    causal = (chunk, 0)
    idx = torch.empty(B, H, nb, k_keep, dtype=torch.int32, device=dev)
    cnt = torch.empty(B, H, nb, dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(B, H, N, dtype=torch.float32, device=dev)
    desc = sa.make_desc(q, k, v, o, block=block, causal=causal)
    ws_sel = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SELECT, k_keep),
                         dtype=torch.uint8, device=dev)
    ws_sch = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SCHEDULE, k_keep),
                         dtype=torch.uint8, device=dev)
    order = torch.empty(sa.sparse_attn_num_tiles(desc), dtype=torch.int32, device=dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]

    def step(e=None):
        if e:
            e[0].record()
        sa.sparse_attn_select(q, k, k_keep, block=block, idx=idx, cnt=cnt, ws=ws_sel,
                              causal=causal)
        if e:
            e[1].record()
        sa.sparse_attn_schedule(cnt, N, k_keep, block=block, order=order, ws=ws_sch)
        if e:
            e[2].record()
        sa.sparse_attn_fwd(q, k, v, idx, cnt, block=block, order=order, o=o, lse=lse,
                           causal=causal)
        if e:
            e[3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for s_ in range(args.steps):
        step(ev[s_])
    torch.cuda.synchronize()
    ms = [float(np.mean([e[i].elapsed_time(e[i + 1]) for e in ev])) for i in range(3)]
    flops = selected_flops(cnt.cpu().numpy(), idx.cpu().numpy(), N, block, d)
    tf = flops / (ms[2] * 1e-3) / 1e12
    return {
        "chunk_tokens": chunk, "window_chunks": 0,
        "ms_per_call": {"select": round(ms[0], 4), "schedule": round(ms[1], 4),
                        "fwd": round(ms[2], 4)},
        "ms_per_step": round(sum(ms), 4),
        "mean_kept_blocks": round(float(cnt.float().mean().item()), 2),
        "roofline": {"kernel": "fwd_bf16_kernel", "bound": "mfma", "achieved": round(tf, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "flops_per_launch": flops,
                     "note": "flops of the selected blocks; masked pairs counted"},
    }


def bench_bwd(args, sa, dev, wl, q, k, v, o, lse, idx, cnt):
    """Backward of the sparse branch at the layer's shape and lists: the
    forward's O and LSE, a seeded normal upstream gradient.  One call runs
    D = rowsum(dO o O), the transposed selection bitmap, the dQ kernel (S, dP
    and dQ products per query tile) and the dK/dV kernel (S, dP, dV and dK
    products per key tile): 7 products of the forward's 2-product size.  The
    algorithmic count is 5 products (S, dP, dV, dK, dQ: 2.5x the forward)."""
    B, H, N, d, block = wl.batch, wl.heads, wl.seqlen, wl.head_dim, wl.block
    g = torch.Generator(device=dev).manual_seed(11)
    do = torch.randn(q.shape, generator=g, device=dev).to(torch.bfloat16)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    desc = sa.make_desc(q, k, v, o, block=block)
    ws = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_BWD, idx.shape[-1]),
                     dtype=torch.uint8, device=dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(args.steps)]

    def step(e=None):
        if e:
            e[0].record()
        sa.sparse_attn_bwd(q, k, v, o, do, lse, idx, cnt, block=block, dq=dq, dk=dk, dv=dv, ws=ws)
        if e:
            e[1].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for s_ in range(args.steps):
        step(ev[s_])
    torch.cuda.synchronize()
    ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    fwd_flops = selected_flops(cnt.cpu().numpy(), idx.cpu().numpy(), N, block, d)
    alg = fwd_flops * 5 // 2
    tf = alg / (ms * 1e-3) / 1e12
    return {
        "ms_per_call": round(ms, 4),
        "executed_tflops": round(fwd_flops * 7 / 2 / (ms * 1e-3) / 1e12, 2),
        "roofline": {"kernel": "bwd (dot, bitmap, dq, dkdv)", "bound": "mfma",
                     "achieved": round(tf, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "flops_per_launch": alg,
                     "note": "algorithmic flops: 2.5x the forward's over the selected blocks"},
    }


def bench_path(args, sa, W, dev, name):
    """select + schedule + fwd (bf16, row top-k) on another workload: ms per
    call (warm median, and cold with the caches flushed before each call) and
    the forward's roofline over the selected blocks."""
    wl = W.WORKLOADS[name]
    B, H, N, d, block = wl.batch, wl.heads, wl.seqlen, wl.head_dim, wl.block
    nb = -(-N // block)
    kk = sa.sparse_attn_keep_count(wl.keep_bp, nb)
    q, k, v = (t.to(dev) for t in W.make_inputs(wl))
    idx = torch.empty(B, H, nb, kk, dtype=torch.int32, device=dev)
    cnt = torch.empty(B, H, nb, dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(B, H, N, dtype=torch.float32, device=dev)
    desc = sa.make_desc(q, k, v, o, block=block)
    ws_sel = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SELECT, kk),
                         dtype=torch.uint8, device=dev)
    ws_sch = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SCHEDULE, kk),
                         dtype=torch.uint8, device=dev)
    order = torch.empty(sa.sparse_attn_num_tiles(desc), dtype=torch.int32, device=dev)
    phases = [
        ("select", lambda: sa.sparse_attn_select(q, k, kk, block=block, idx=idx, cnt=cnt,
                                                 ws=ws_sel)),
        ("schedule", lambda: sa.sparse_attn_schedule(cnt, N, kk, block=block, order=order,
                                                     ws=ws_sch)),
        ("fwd", lambda: sa.sparse_attn_fwd(q, k, v, idx, cnt, block=block, order=order, o=o,
                                           lse=lse)),
    ]
    warm = time_calls(phases, args.steps, args.warmup)
    cold = time_calls(phases, max(3, args.steps // 2), 1, flush=args.flusher)
    flops = selected_flops(cnt.cpu().numpy(), idx.cpu().numpy(), N, block, d)
    dense = 4 * B * H * N * N * d
    fwd_ms = med(warm["fwd"])
    tf = flops / (fwd_ms * 1e-3) / 1e12
    step_ms = sum(med(warm[n]) for n, _ in phases)
    return {
        "workload": name, "generator": wl.gen,
        "shape": {"batch": B, "heads": H, "seqlen": N, "grid": list(wl.grid), "block": block,
                  "keep_blocks": kk, "key_blocks": nb},
        "ms_per_call": {n: med(warm[n]) for n, _ in phases},
        "ms_per_call_cold": {n: med(cold[n]) for n, _ in phases},
        "ms_per_step": round(step_ms, 4),
        "dense_equiv_tflops_step": round(dense / (step_ms * 1e-3) / 1e12, 2),
        "roofline": {"kernel": "fwd_bf16_kernel", "bound": "mfma", "achieved": round(tf, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / PEAK_BF16_TFLOPS, 4), "traffic": None,
                     "flops_per_launch": flops},
    }


def bench_sweep(args, sa, W, dev):
    """select + schedule + fwd (bf16, row top-k) at every point of the
    sparsity sweep on the locality inputs (40 heads x 75,600 tokens): ms per
    call and the forward's actual TFLOP/s over the selected blocks."""
    wl = W.WORKLOADS["sweep"]
    B, H, N, d = wl.batch, wl.heads, wl.seqlen, wl.head_dim
    q, k, v = (t.to(dev) for t in W.make_inputs(wl))
    o = torch.empty_like(q)
    lse = torch.empty(B, H, N, dtype=torch.float32, device=dev)
    dense = 4 * B * H * N * N * d
    steps, warm = min(args.steps, 5), min(args.warmup, 2)
    points = []
    for block, keep in wl.sweep:
        nb = -(-N // block)
        kk = sa.sparse_attn_keep_count(keep, nb)
        idx = torch.empty(B, H, nb, kk, dtype=torch.int32, device=dev)
        cnt = torch.empty(B, H, nb, dtype=torch.int32, device=dev)
        desc = sa.make_desc(q, k, v, o, block=block)
        ws_sel = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SELECT, kk),
                             dtype=torch.uint8, device=dev)
        ws_sch = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SCHEDULE, kk),
                             dtype=torch.uint8, device=dev)
        order = torch.empty(sa.sparse_attn_num_tiles(desc), dtype=torch.int32, device=dev)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(steps)]

        def step(e=None):
            if e:
                e[0].record()
            sa.sparse_attn_select(q, k, kk, block=block, idx=idx, cnt=cnt, ws=ws_sel)
            if e:
                e[1].record()
            sa.sparse_attn_schedule(cnt, N, kk, block=block, order=order, ws=ws_sch)
            if e:
                e[2].record()
            sa.sparse_attn_fwd(q, k, v, idx, cnt, block=block, order=order, o=o, lse=lse)
            if e:
                e[3].record()

        for _ in range(warm):
            step()
        torch.cuda.synchronize()
        for s_ in range(steps):
            step(ev[s_])
        torch.cuda.synchronize()
        ms = [float(np.mean([e[i].elapsed_time(e[i + 1]) for e in ev])) for i in range(3)]
        flops = selected_flops(cnt.cpu().numpy(), idx.cpu().numpy(), N, block, d)
        tf = flops / (ms[2] * 1e-3) / 1e12
        points.append({"block": block, "keep": keep / 10000, "k": kk, "key_blocks": nb,
                       "ms_per_call": {"select": round(ms[0], 4), "schedule": round(ms[1], 4),
                                       "fwd": round(ms[2], 4)},
                       "fwd_actual_tflops": round(tf, 2),
                       "fwd_mfma_frac": round(tf / PEAK_BF16_TFLOPS, 4),
                       "step_dense_equiv_tflops": round(dense / (sum(ms) * 1e-3) / 1e12, 2)})
        del idx, cnt, ws_sel, ws_sch, order
    return {"workload": wl.name, "generator": wl.gen, "steps": steps, "points": points}


def bench_linear(args, sa, W, dev):
    """W8A8 fp8 linear layer at the 14B-720P projection shape (75,600 tokens,
    5120 -> 5120): per-token e4m3 quantisation of the bf16 activations in one
    pass, then the fp8 GEMM with per-token x per-channel scales and bias to a
    bf16 output.  The weights are quantised once beforehand (offline in the
    paper) and not timed.  A library fp8 GEMM with the same row-wise scales
    (torch._scaled_mm, hipBLASLt) is timed beside it for context when
    available."""
    name = "wan14b_720p_qkvo"
    M, K, N = W.LINEAR_SHAPES[name]
    g = torch.Generator(device=dev)
    g.manual_seed(7)
    x = torch.randn(M, K, device=dev, generator=g)
    x[:, :max(1, K // 1000)] *= 20.0                   # channel outliers
    x = x.to(torch.bfloat16)
    w = (torch.randn(N, K, device=dev, generator=g) / K ** 0.5).to(torch.bfloat16)
    bias = 0.1 * torch.randn(N, device=dev, generator=g)
    wq, sw = sa.sparse_attn_quant_rows_fp8(w)
    xq = torch.empty(M, K, dtype=torch.uint8, device=dev)
    sx = torch.empty(M, dtype=torch.float32, device=dev)
    y = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]

    def step(e=None):
        if e:
            e[0].record()
        sa.sparse_attn_quant_rows_fp8(x, xq, sx)
        if e:
            e[1].record()
        sa.sparse_attn_linear_w8a8(xq, sx, wq, sw, bias, y)
        if e:
            e[2].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    for s_ in range(args.steps):
        step(ev[s_])
    torch.cuda.synchronize()
    q_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    g_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    flops = 2.0 * M * N * K
    q_bytes = M * K * 2 + M * K + M * 4
    g_tf = flops / (g_ms * 1e-3) / 1e12
    out = {
        "shape": {"tokens": M, "in_features": K, "out_features": N},
        "ms_per_call": {"quant_rows_fp8": round(q_ms, 4), "linear_w8a8": round(g_ms, 4)},
        "ms_per_layer": round(q_ms + g_ms, 4),
        "roofline": {
            "kernel": "linear_w8a8_kernel", "bound": "mfma", "achieved": round(g_tf, 1),
            "peak": PEAK_FP8_TFLOPS, "unit": "TFLOP/s", "frac": round(g_tf / PEAK_FP8_TFLOPS, 4),
            "traffic": None, "flops_per_launch": flops,
        },
        "quant_roofline": {
            "kernel": "quant_rows_kernel", "bound": "hbm",
            "achieved": round(q_bytes / (q_ms * 1e-3) / 1e9, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(q_bytes / (q_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "traffic": None, "algorithmic_bytes_per_launch": q_bytes,
        },
    }
    try:
        f = lambda: torch._scaled_mm(xq.view(torch.float8_e4m3fn),
                                     wq.view(torch.float8_e4m3fn).t(),
                                     scale_a=sx.view(-1, 1), scale_b=sw.view(1, -1),
                                     bias=None, out_dtype=torch.bfloat16)
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            f()
        e1.record()
        torch.cuda.synchronize()
        lib_ms = e0.elapsed_time(e1) / args.steps
        out["library_fp8_gemm"] = {"what": "torch._scaled_mm (hipBLASLt), row-wise scales, "
                                           "no bias", "ms": round(lib_ms, 4),
                                   "tflops": round(flops / (lib_ms * 1e-3) / 1e12, 1)}
    except Exception as exc:  # pragma: no cover - depends on the torch build
        out["library_fp8_gemm"] = {"error": str(exc)[:120]}
    return out


def bench_fp8(args, sa, W, dev):
    """fp8 pass at the same shape on the outlier workload: bf16 selection,
    e4m3 quantisation of Q, K, V, scheduling, fp8 fused forward."""
    wl = W.WORKLOADS["wan14b_720p_fp8"]
    B, H, N, d, block = wl.batch, wl.heads, wl.seqlen, wl.head_dim, wl.block
    nb = -(-N // block)
    k = sa.sparse_attn_keep_count(wl.keep_bp, nb)
    q, kk, v = (t.to(dev) for t in W.make_inputs(wl))
    idx = torch.empty(B, H, nb, k, dtype=torch.int32, device=dev)
    cnt = torch.empty(B, H, nb, dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(B, H, N, dtype=torch.float32, device=dev)
    # Q row-major, K and V in the forward's tile layouts
    x8 = [torch.empty(B, H, N, d, dtype=torch.uint8, device=dev)] + \
        [torch.empty(B, H, -(-N // 64), 8192, dtype=torch.uint8, device=dev) for _ in range(2)]
    sc = [torch.empty(B, H, nb, dtype=torch.float32, device=dev) for _ in range(3)]
    desc = sa.make_desc(q, kk, v, o, block=block)
    ws_sel = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SELECT, k),
                         dtype=torch.uint8, device=dev)
    ws_sch = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SCHEDULE, k),
                         dtype=torch.uint8, device=dev)
    order = torch.empty(sa.sparse_attn_num_tiles(desc), dtype=torch.int32, device=dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]

    def step(e=None):
        if e:
            e[0].record()
        sa.sparse_attn_select(q, kk, k, block=block, idx=idx, cnt=cnt, ws=ws_sel)
        if e:
            e[1].record()
        sa.sparse_attn_quant_fp8(q, block=block, x8=x8[0], scale=sc[0])
        sa.sparse_attn_quant_fp8_tiles(kk, sa.SA_FP8_K, block=block, x8=x8[1], scale=sc[1])
        sa.sparse_attn_quant_fp8_tiles(v, sa.SA_FP8_V, block=block, x8=x8[2], scale=sc[2])
        if e:
            e[2].record()
        sa.sparse_attn_schedule(cnt, N, k, block=block, order=order, ws=ws_sch)
        if e:
            e[3].record()
        sa.sparse_attn_fwd_fp8(x8[0], sc[0], x8[1], sc[1], x8[2], sc[2], idx, cnt, block=block,
                               order=order, o=o, lse=lse)
        if e:
            e[4].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(ev[s])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    ms = [float(np.mean([e[i].elapsed_time(e[i + 1]) for e in ev])) for i in range(4)]
    flops = selected_flops(cnt.cpu().numpy(), idx.cpu().numpy(), N, block, d)
    dense = 4 * B * H * N * N * d
    tf = flops / (ms[3] * 1e-3) / 1e12
    qbytes = 3 * (B * H * N * d * 3 + B * H * nb * 4)   # bf16 in, e4m3 out, scales
    return {
        "workload": wl.name, "dtype": "fp8-e4m3", "ms_per_step": round(ms_step, 4),
        "dense_equiv_tflops_step": round(dense / (ms_step * 1e-3) / 1e12, 2),
        "ms_per_call": {"select": round(ms[0], 4), "quant_qkv": round(ms[1], 4),
                        "schedule": round(ms[2], 4), "fwd_fp8": round(ms[3], 4)},
        "fwd_actual_tflops": round(tf, 2), "fwd_mfma_frac": round(tf / PEAK_FP8_TFLOPS, 4),
        "quant_gbs": round(qbytes / (ms[1] * 1e-3) / 1e9, 1),
        "roofline": {"kernel": "fwd_fp8_kernel", "bound": "mfma", "achieved": round(tf, 2),
                     "peak": PEAK_FP8_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(tf / PEAK_FP8_TFLOPS, 4),
                     "traffic": measured_traffic("fwd_fp8_kernel", wl.name),
                     "flops_per_launch": flops},
    }


def main():
    args = parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import paper_2609_23153_amd as sa
    import workloads as W

    wl = W.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    B, H, N, d, block = wl.batch, wl.heads, wl.seqlen, wl.head_dim, wl.block
    nb = -(-N // block)
    k = sa.sparse_attn_keep_count(wl.keep_bp, nb)

    log(f"generating {wl.name}")
    q, kk, v = (t.to(dev) for t in W.make_inputs(wl))
    idx = torch.empty(B, H, nb, k, dtype=torch.int32, device=dev)
    cnt = torch.empty(B, H, nb, dtype=torch.int32, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(B, H, N, dtype=torch.float32, device=dev)
    desc = sa.make_desc(q, kk, v, o, block=block)
    ws_sel = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SELECT, k),
                         dtype=torch.uint8, device=dev)
    ws_sch = torch.empty(sa.sparse_attn_workspace_size(desc, sa.SA_OP_SCHEDULE, k),
                         dtype=torch.uint8, device=dev)
    order = torch.empty(sa.sparse_attn_num_tiles(desc), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()

    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]

    def step(e=None):
        if e:
            e[0].record()
        sa.sparse_attn_select(q, kk, k, block=block, idx=idx, cnt=cnt, ws=ws_sel)
        if e:
            e[1].record()
        sa.sparse_attn_schedule(cnt, N, k, block=block, order=order, ws=ws_sch)
        if e:
            e[2].record()
        sa.sparse_attn_fwd(q, kk, v, idx, cnt, block=block, order=order, o=o, lse=lse)
        if e:
            e[3].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(ev[s])
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    ms_step = (t1 - t0) * 1e3 / args.steps
    sel_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    sch_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    fwd_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in ev]))

    args.flusher = CacheFlush(dev) if args.cold == "on" else None
    phases = [
        ("select", lambda: sa.sparse_attn_select(q, kk, k, block=block, idx=idx, cnt=cnt,
                                                 ws=ws_sel)),
        ("schedule", lambda: sa.sparse_attn_schedule(cnt, N, k, block=block, order=order,
                                                     ws=ws_sch)),
        ("fwd", lambda: sa.sparse_attn_fwd(q, kk, v, idx, cnt, block=block, order=order, o=o,
                                           lse=lse)),
    ]
    timing = {"warm_median_ms": {n: med([e[i].elapsed_time(e[i + 1]) for e in ev])
                                 for i, (n, _) in enumerate(phases)}}
    if args.flusher is not None:
        cold = time_calls(phases, args.steps, 1, flush=args.flusher)
        cold_step = time_calls([("step", step)], args.steps, 0, flush=args.flusher)["step"]
        timing["cold_median_ms"] = {n: med(cold[n]) for n, _ in phases}
        timing["cold_step_median_ms"] = med(cold_step)
        timing["cold_note"] = ("a 512 MB device buffer is overwritten before every timed call "
                               "(and before every timed step), so L2 and the Infinity Cache "
                               "hold none of its inputs; medians of HIP-event times")

    flops = selected_flops(cnt.cpu().numpy(), idx.cpu().numpy(), N, block, d)
    dense = 4 * B * H * N * N * d
    fwd_tflops = flops / (fwd_ms * 1e-3) / 1e12
    sel_bytes = 2 * B * H * N * d * 2 + B * H * nb * (k + 1) * 4
    out = {
        "metric": METRIC,
        "value": round(dense / (ms_step * 1e-3) / 1e12, 2),
        "unit": "dense-equiv TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": wl.name, "batch": B, "heads": H, "seqlen": N, "grid": list(wl.grid),
            "head_dim": d, "block": block, "keep_blocks": k, "key_blocks": nb,
            "sparsity": round(1 - k / nb, 4), "generator": wl.gen,
        },
        "ms_per_call": {"select": round(sel_ms, 4), "schedule": round(sch_ms, 4),
                        "fwd": round(fwd_ms, 4)},
        "fwd_actual_tflops": round(fwd_tflops, 2),
        "fwd_dense_equiv_tflops": round(dense / (fwd_ms * 1e-3) / 1e12, 2),
        "fwd_mfma_frac": round(fwd_tflops / PEAK_BF16_TFLOPS, 4),
        "select_gbs": round(sel_bytes / (sel_ms * 1e-3) / 1e9, 1),
        "select_roofline": {
            "kernels": ["pool_kernel", "score_topk_kernel"], "bound": "hbm",
            "achieved": round(sel_bytes / (sel_ms * 1e-3) / 1e9, 1), "peak": PEAK_HBM_GBS,
            "unit": "GB/s", "frac": round(sel_bytes / (sel_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            "traffic": sel_traffic(wl.name), "algorithmic_bytes_per_call": sel_bytes,
            "note": "Q and K read once, lists written; the whole selection call"},
        "timing": timing,
        "roofline": {
            "kernel": "fwd_bf16_kernel", "bound": "mfma",
            "achieved": round(fwd_tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": round(fwd_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": measured_traffic("fwd_bf16_kernel", wl.name),
            "flops_per_launch": flops,
            "algorithmic_bytes_per_launch": 4 * B * H * N * d * 2 + B * H * N * 4
                                            + B * H * nb * (k + 1) * 4,
        },
    }

    log(f"headline step {ms_step:.3f} ms (fwd {fwd_ms:.3f} ms)")
    if args.comp == "on":
        log("compensation")
        out["compensation"] = bench_comp(args, sa, W, dev, wl, q, kk, v, o, ms_step)
    if args.fp8 == "on":
        log("fp8")
        out["fp8"] = bench_fp8(args, sa, W, dev)
    if args.causal == "on":
        log("causal")
        out["causal"] = bench_causal(args, sa, W, dev, wl, q, kk, v)
    if args.bwd == "on":
        log("backward")
        out["backward"] = bench_bwd(args, sa, dev, wl, q, kk, v, o, lse, idx, cnt)
    if args.linear == "on":
        log("linear")
        out["linear_w8a8"] = bench_linear(args, sa, W, dev)
    if args.wan13b == "on":
        log("wan13b_480p")
        out["wan13b_480p"] = bench_path(args, sa, W, dev, "wan13b_480p")
    if args.normal == "on":
        log("wan14b_720p_normal")
        out["wan14b_720p_normal"] = bench_path(args, sa, W, dev, "wan14b_720p_normal")
    if args.sweep == "on":
        log("sweep")
        out["sweep"] = bench_sweep(args, sa, W, dev)

    if args.copy_calib:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        bb = torch.empty_like(a)
        for _ in range(3):
            bb.copy_(a)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(5):
            bb.copy_(a)
        e1.record()
        torch.cuda.synchronize()
        out["copy_calib"] = {"bytes_each_way": 1 << 30, "ms": e0.elapsed_time(e1) / 5}

    if args.cpu_baseline == "on":
        log("cpu baseline")
        import oracle as O
        tau = W.softmax_scale(d)
        nh = max(1, min(args.cpu_heads, H))
        sample = sorted({int(round(i * (H - 1) / max(1, nh - 1))) for i in range(nh)})
        t_sel = t_fwd = 0.0
        for h in sample:
            log(f"  oracle head {h}")
            qf, kf, vf = (t.to(torch.float64).numpy() for t in W.make_head(wl, 0, h))
            t0 = time.perf_counter()
            ri, rc = O.select_head(qf, kf, block, wl.keep_bp)
            t1 = time.perf_counter()
            O.sparse_attention(qf, kf, vf, ri, rc, block, tau)
            t2 = time.perf_counter()
            t_sel += t1 - t0
            t_fwd += t2 - t1
        scale_h = (B * H) / len(sample)
        per_call = (t_sel + t_fwd) * scale_h
        out["cpu_baseline"] = {
            "value": round(dense / per_call / 1e12, 6),
            "unit": "dense-equiv TFLOP/s",
            "ms_per_call": round(per_call * 1e3, 1),
            "ms_per_call_select": round(t_sel * scale_h * 1e3, 1),
            "ms_per_call_fwd": round(t_fwd * scale_h * 1e3, 1),
            "cores": blas_threads(),
            "cpu_model": cpu_model(),
            "kind": "oracle",
            "sample": f"fp64 NumPy oracle, select + attention of {len(sample)} of {H} heads "
                      f"{sample} ({t_sel + t_fwd:.1f} s: select {t_sel:.1f} s, attention "
                      f"{t_fwd:.1f} s), scaled x{scale_h:g} to the full layer",
        }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()

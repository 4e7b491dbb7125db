"""Host-side checks of the C ABI: the library loads, exports every function
the header declares, and rejects invalid arguments before any HIP call (so
these run without a GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2609_23153_amd as sa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparse_attn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sparse_attn_\w+)\s*\(", text)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(sa.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", sa.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT\s+(\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(sa.library(), name)


def test_version_status_keep_count():
    assert sa.sparse_attn_version() == 100
    assert sa.sparse_attn_status_str(0) == "ok"
    assert sa.sparse_attn_status_str(-3) == "workspace too small"
    assert sa.sparse_attn_status_str(12345) == "unknown status"
    assert sa.sparse_attn_keep_count(1000, 64) == 7
    assert sa.sparse_attn_keep_count(300, 1182) == 36
    assert sa.sparse_attn_keep_count(10000, 591) == 591
    assert sa.sparse_attn_keep_count(1, 10) == 1
    assert sa.sparse_attn_keep_count(0, 10) == -1


def desc(B=1, H=2, N=4096, d=128, block=64, scale=0.0):
    ds = sa.SparseAttnDesc()
    ds.batch, ds.heads, ds.seqlen, ds.head_dim, ds.block = B, H, N, d, block
    st = (H * N * d, N * d, d)
    for f in ("q_stride", "k_stride", "v_stride", "o_stride"):
        getattr(ds, f)[:] = st
    ds.softmax_scale = scale
    return ds


def test_workspace_size_formula():
    lib = sa.library()
    ds = desc(B=1, H=40, N=75600)
    nb = 1182
    # row mode: pooled q/k (fp64), the bf16 hi/lo operand of the pooled keys
    # for the on-chip scores in tiles of 32 blocks (16 KB per tile), fp32 key
    # norms (the query side is pooled on chip)
    assert lib.sparse_attn_workspace_size(ctypes.byref(ds), 0, 36) == \
        40 * nb * 128 * 8 * 2 + 40 * 37 * 16384 + 40 * nb * 4
    # whole-head mode: pooled q/k, scores (fp64), then per head 32 B of radix
    # state and a 256-bin histogram, per row 3 int32
    assert lib.sparse_attn_workspace_size(ctypes.byref(ds), sa.SA_OP_SELECT_HEAD, 36) == \
        40 * nb * 128 * 8 * 2 + 40 * nb * nb * 8 + 40 * 32 + 40 * 256 * 4 + 3 * 40 * nb * 4
    # row mode past 1192 blocks: pooled q/k and the fp64 score matrix
    big = desc(B=1, H=2, N=1193 * 64)
    assert lib.sparse_attn_workspace_size(ctypes.byref(big), 0, 36) == \
        2 * 1193 * 128 * 8 * 2 + 2 * 1193 * 1193 * 8
    edge = desc(B=1, H=2, N=1192 * 64)
    assert lib.sparse_attn_workspace_size(ctypes.byref(edge), 0, 36) == \
        2 * 1192 * 128 * 8 * 2 + 2 * 38 * 16384 + 2 * 1192 * 4
    # scheduler: 16 class counters per chunk of 1024 query tiles, plus one row
    assert lib.sparse_attn_workspace_size(ctypes.byref(ds), 1, 36) == (47 + 1) * 16 * 4
    assert lib.sparse_attn_workspace_size(ctypes.byref(ds), 1, 0) == 0
    assert lib.sparse_attn_workspace_size(ctypes.byref(ds), 7, 36) == 0
    assert lib.sparse_attn_workspace_size(ctypes.byref(desc(d=64)), 0, 1) == 0
    assert lib.sparse_attn_workspace_size(None, 0, 1) == 0


def test_tile_count_limit():
    # B*H*ceil(L/64) query tiles must stay <= 2^30 (32-bit tile indices), also
    # when B*H*nkb does (block 128 halves nkb but not the 64-row tiles)
    lib = sa.library()
    assert lib.sparse_attn_num_tiles(ctypes.byref(desc(H=131072, N=524288, block=128))) == \
        131072 * 8192
    assert lib.sparse_attn_num_tiles(ctypes.byref(desc(H=131073, N=524288, block=128))) == -1


# Fake, aligned, non-null device addresses: every call below must fail its
# host-side checks, so nothing is ever dereferenced or launched.
P = ctypes.c_void_p(1 << 20)
MIS = ctypes.c_void_p((1 << 20) + 2)
WS = 1 << 40


@pytest.mark.parametrize("case,expect", [
    (dict(d=64), -2), (dict(block=32), -2), (dict(block=256), -2), (dict(N=0), -1),
    (dict(B=0), -1), (dict(H=-1), -1), (dict(scale=-1.0), -1), (dict(scale=float("nan")), -1),
    (dict(N=64 * 4097), -2),
])
def test_select_rejects_bad_descriptors(case, expect):
    lib = sa.library()
    ds = desc(**case)
    st = lib.sparse_attn_select(ctypes.byref(ds), P, P, 0, 7, P, P, 7, P, WS, None)
    assert st == expect


def test_select_rejects_bad_arguments():
    lib = sa.library()
    ds = desc()
    call = lambda *a: lib.sparse_attn_select(ctypes.byref(ds), *a)
    assert call(None, P, 0, 7, P, P, 7, P, WS, None) == -1          # null q
    assert call(P, P, 0, 7, None, P, 7, P, WS, None) == -1          # null idx
    assert call(MIS, P, 0, 7, P, P, 7, P, WS, None) == -1           # misaligned q
    assert call(P, P, 0, 0, P, P, 7, P, WS, None) == -1             # topk 0
    assert call(P, P, 0, 65, P, P, 65, P, WS, None) == -1           # topk > nkb
    assert call(P, P, 0, 7, P, P, 6, P, WS, None) == -1             # kmax < topk
    assert call(P, P, 9, 7, P, P, 7, P, WS, None) == -1             # bad mode
    assert call(P, P, 1, 63, P, P, 7, P, WS, None) == -1            # head budget < nqb
    assert call(P, P, 1, 64 * 64 + 1, P, P, 7, P, WS, None) == -1   # head budget > nqb*nkb
    assert call(P, P, 0, 7, P, P, 7, P, 100, None) == -3            # workspace too small
    # each mode checks against its own size (at 1182 blocks the whole-head
    # mode's score matrix makes it the larger)
    big = desc(N=75600)
    row = lib.sparse_attn_workspace_size(ctypes.byref(big), sa.SA_OP_SELECT, 7)
    head = lib.sparse_attn_workspace_size(ctypes.byref(big), sa.SA_OP_SELECT_HEAD, 7)
    assert 0 < row < head
    sel = lambda *a: lib.sparse_attn_select(ctypes.byref(big), *a)
    assert sel(P, P, 0, 7, P, P, 7, P, row - 1, None) == -3
    assert sel(P, P, 1, 5000, P, P, 64, P, row, None) == -3
    assert sel(P, P, 1, 5000, P, P, 64, P, head - 1, None) == -3
    ds.q_stride[2] = 130                                            # stride not multiple of 8
    assert call(P, P, 0, 7, P, P, 7, P, WS, None) == -1


def test_fwd_rejects_bad_arguments():
    lib = sa.library()
    ds = desc()
    call = lambda *a: lib.sparse_attn_fwd(ctypes.byref(ds), *a)
    assert call(None, P, P, P, P, 7, None, P, None, None) == -1     # null q
    assert call(P, P, P, None, P, 7, None, P, None, None) == -1     # null idx
    assert call(P, P, P, P, None, 7, None, P, None, None) == -1     # null cnt
    assert call(P, P, P, P, P, 0, None, P, None, None) == -1        # kmax 0
    assert call(P, P, P, P, P, 7, None, MIS, None, None) == -1      # misaligned o
    assert call(P, P, P, P, P, 7, None, None, None, None) == -1     # null o
    ds.v_stride[1] = 12                                              # stride not multiple of 8
    assert call(P, P, P, P, P, 7, None, P, None, None) == -1
    ds.head_dim = 96
    assert call(P, P, P, P, P, 7, None, P, None, None) == -2


def test_schedule_rejects_bad_arguments():
    lib = sa.library()
    ds = desc(B=2, H=3, N=1000)
    assert lib.sparse_attn_num_tiles(ctypes.byref(ds)) == 2 * 3 * 16
    assert lib.sparse_attn_num_tiles(ctypes.byref(desc(block=96))) == -1
    need = lib.sparse_attn_workspace_size(ctypes.byref(ds), 1, 7)
    assert need == (1 + 1) * 16 * 4                                   # one chunk of 96 tiles
    call = lambda *a: lib.sparse_attn_schedule(ctypes.byref(ds), *a)
    assert call(None, 7, P, P, need, None) == -1                    # null cnt
    assert call(P, 7, None, P, need, None) == -1                    # null order
    assert call(P, 0, P, P, need, None) == -1                       # kmax 0
    assert call(P, 7, P, P, need - 1, None) == -3                   # workspace


def test_quant_and_fwd_fp8_reject_bad_arguments():
    lib = sa.library()
    ds = desc()
    st3 = (ctypes.c_int64 * 3)(2 * 4096 * 128, 4096 * 128, 128)
    assert lib.sparse_attn_quant_fp8(ctypes.byref(ds), None, st3, P, P, None) == -1
    assert lib.sparse_attn_quant_fp8(ctypes.byref(ds), P, None, P, P, None) == -1
    assert lib.sparse_attn_quant_fp8(ctypes.byref(ds), MIS, st3, P, P, None) == -1
    bad = (ctypes.c_int64 * 3)(2 * 4096 * 128, 4096 * 128, 129)
    assert lib.sparse_attn_quant_fp8(ctypes.byref(ds), P, bad, P, P, None) == -1
    qt = lambda *a: lib.sparse_attn_quant_fp8_tiles(ctypes.byref(ds), *a)
    assert qt(None, st3, sa.SA_FP8_K, P, P, None) == -1             # null x
    assert qt(P, st3, 2, P, P, None) == -1                          # bad operand
    assert qt(P, st3, sa.SA_FP8_V, MIS, P, None) == -1              # misaligned x8
    assert qt(P, bad, sa.SA_FP8_K, P, P, None) == -1                # bad stride
    assert lib.sparse_attn_fp8_tiles_bytes(ctypes.byref(ds)) == 2 * 64 * 8192
    assert lib.sparse_attn_fp8_tiles_bytes(ctypes.byref(desc(N=4097))) == 2 * 65 * 8192
    assert lib.sparse_attn_fp8_tiles_bytes(ctypes.byref(desc(d=64))) == -1
    f = lambda *a: lib.sparse_attn_fwd_fp8(ctypes.byref(ds), *a)
    assert f(P, None, P, P, P, P, P, P, 7, None, P, None, None) == -1    # null sq
    assert f(P, P, P, P, P, P, P, P, 0, None, P, None, None) == -1       # kmax 0
    assert f(P, P, P, P, P, P, None, P, 7, None, P, None, None) == -1    # null idx
    assert f(P, P, MIS, P, P, P, P, P, 7, None, P, None, None) == -1     # misaligned k8


def test_comp_entry_points_reject_bad_arguments():
    lib = sa.library()
    ds = desc(B=1, H=2, N=4096)
    st3 = (ctypes.c_int64 * 3)(2 * 4096 * 128, 4096 * 128, 128)
    need = lib.sparse_attn_workspace_size(ctypes.byref(ds), sa.SA_OP_COMP_STATE, 1)
    assert need == 1 * 2 * 4 * 64 * 128 * 4          # 4 chunks of 1024 tokens per head
    cs = lambda *a: lib.sparse_attn_comp_state(ctypes.byref(ds), *a)
    assert cs(32, P, st3, P, P, P, P, P, need, None) == -2          # rank must be 64
    assert cs(64, None, st3, P, P, P, P, P, need, None) == -1       # null k_norm
    assert cs(64, MIS, st3, P, P, P, P, P, need, None) == -1        # misaligned
    assert cs(64, P, None, P, P, P, P, P, need, None) == -1         # null strides
    assert cs(64, P, st3, P, P, P, P, P, need - 1, None) == -3      # workspace
    co = lambda *a: lib.sparse_attn_comp_out(ctypes.byref(ds), *a)
    g3 = (ctypes.c_int64 * 3)(2 * 4096, 4096, 1)
    bad_g3 = (ctypes.c_int64 * 3)(2 * 4096, -4096, 1)
    assert co(16, P, st3, P, P, P, None, 1e-6, P, g3, P, P, None) == -2      # rank
    assert co(64, P, st3, P, P, P, None, 1e-6, None, g3, P, P, None) == -1   # null gate
    assert co(64, P, st3, P, P, P, None, -1.0, P, g3, P, P, None) == -1      # eps < 0
    assert co(64, P, st3, P, P, P, None, 1e-6, P, bad_g3, P, P, None) == -1  # gate stride
    assert co(64, P, st3, P, P, P, MIS, 1e-6, P, g3, P, P, None) == -1       # gamma misaligned


def test_w8a8_linear_entry_points_reject_bad_arguments():
    lib = sa.library()
    q = lib.sparse_attn_quant_rows_fp8
    assert q(None, 4, 64, 64, P, P, None) == -1          # null x
    assert q(P, 4, 60, 64, P, P, None) == -1             # cols % 8
    assert q(P, 4, 64, 32, P, P, None) == -1             # ldx < cols
    assert q(P, 4, 64, 68, P, P, None) == -1             # ldx % 8
    assert q(MIS, 4, 64, 64, P, P, None) == -1           # misaligned x
    assert q(P, -1, 64, 64, P, P, None) == -1            # rows < 0
    assert q(P, 0, 64, 64, P, P, None) == 0              # empty: nothing launched
    lin = lib.sparse_attn_linear_w8a8
    ok = (P, P, 256, P, P, 256, None, P, 256, 300, 256, 256, None)

    def call(**kw):
        names = ("xq", "sx", "ldx", "wq", "sw", "ldw", "bias", "y", "ldy", "M", "N", "K", "s")
        args = dict(zip(names, ok))
        args.update(kw)
        return lin(*[args[n] for n in names])

    assert call(M=0) == 0                                # empty: nothing launched
    assert call(N=0, ldy=0) == 0
    assert call(xq=None) == -1
    assert call(sw=None) == -1
    assert call(K=320, ldx=384, ldw=384) == -1           # K % 128
    assert call(K=192, ldx=192, ldw=192) == -1           # K < 256
    assert call(K=0) == -1
    assert call(N=260, ldy=264) == -1                    # N % 8
    assert call(ldx=240) == -1                           # ldx < K
    assert call(ldw=136) == -1                           # ldw % 16
    assert call(ldy=255) == -1                           # ldy < N
    assert call(ldy=260) == -1                           # ldy % 8
    assert call(y=ctypes.c_void_p((1 << 20) + 8)) == -1  # y not 16-byte aligned
    assert call(wq=MIS) == -1                            # misaligned codes
    assert call(bias=MIS) == -1                          # misaligned bias
    assert call(M=-5) == -1
    assert call(ldx=1 << 24) == -2                       # 256 * ldx does not fit 32 bits


def test_causal_window_fields_are_checked():
    lib = sa.library()
    st3 = (ctypes.c_int64 * 3)(2 * 4096 * 128, 4096 * 128, 128)
    need = lib.sparse_attn_workspace_size(ctypes.byref(desc()), sa.SA_OP_SELECT, 7)

    def sel(chunk, window, mode=sa.SA_SELECT_ROW_TOPK, budget=7):
        ds = desc()
        ds.causal_chunk, ds.causal_window = chunk, window
        return lib.sparse_attn_select(ctypes.byref(ds), P, P, mode, budget, P, P, 64, P, need,
                                      None)

    assert sel(-1, 0) == -1                       # negative chunk
    assert sel(1024, -2) == -1                    # negative window
    assert sel(0, 3) == -1                        # window without chunks
    assert sel(1024, 2, mode=sa.SA_SELECT_HEAD_TOPK, budget=500) == -2   # whole-head mode
    # the compensation state keeps one partial per (chunk, 1024-token
    # sub-chunk) of the 4096 tokens: chunks of 1000 -> 5 x 1 partials, one
    # chunk of 4096 -> 4, chunks of 1500 -> 3 x 2
    d0 = desc()
    base = lib.sparse_attn_workspace_size(ctypes.byref(d0), sa.SA_OP_COMP_STATE, 1)
    for chunk, parts in ((1000, 5), (4096, 4), (1500, 6)):
        ds = desc()
        ds.causal_chunk, ds.causal_window = chunk, 0
        assert lib.sparse_attn_workspace_size(ctypes.byref(ds), sa.SA_OP_COMP_STATE, 1) == \
            base // 4 * parts
    assert ctypes.sizeof(sa.SparseAttnDesc) == 136   # the C struct with the two int32 fields


def test_bwd_rejects_bad_arguments():
    lib = sa.library()
    ds = desc()
    need = lib.sparse_attn_workspace_size(ctypes.byref(ds), sa.SA_OP_BWD, 7)
    assert need > 0

    def call(d=ds, **kw):
        names = ("q", "k", "v", "o", "do", "lse", "idx", "cnt", "kmax", "dq", "dk", "dv", "ws",
                 "wsb")
        args = dict(zip(names, (P, P, P, P, P, P, P, P, 7, P, P, P, P, need)))
        args.update(kw)
        return lib.sparse_attn_bwd(ctypes.byref(d), *[args[n] for n in names], None)

    assert call(q=None) == -1                     # null input
    assert call(do=None) == -1                    # null upstream gradient
    assert call(lse=None) == -1                   # null LSE
    assert call(dv=None) == -1                    # null output
    assert call(ws=None) == -1                    # null workspace
    assert call(idx=None) == -1                   # null list
    assert call(kmax=0) == -1                     # kmax 0
    assert call(dk=MIS) == -1                     # misaligned output
    assert call(o=MIS) == -1                      # misaligned forward output
    assert call(wsb=need - 1) == -3               # workspace too small
    bad = desc()
    bad.o_stride[2] = 132                         # token stride not a multiple of 8
    assert call(d=bad) == -1
    bad = desc(d=64)
    assert call(d=bad) == -2                      # head_dim
    # a token-major layout whose head spans >= 4 GiB: (N + 64) * stride * 2
    # bytes past the 32-bit row offsets of the kernels
    for f in ("q_stride", "k_stride", "v_stride", "o_stride"):
        big = desc(N=75600)
        getattr(big, f)[2] = 28416                # (75600 + 64) * 28416 * 2 >= 2^32
        wsb = lib.sparse_attn_workspace_size(ctypes.byref(big), sa.SA_OP_BWD, 7)
        assert call(d=big, wsb=wsb) == -2, f
        getattr(big, f)[2] = 28368                # just inside: passes the range check
        assert (75600 + 64) * 28368 * 2 + 256 < 1 << 32
    # the forward rejects the same layouts
    big = desc(N=75600)
    big.k_stride[2] = 28416
    assert lib.sparse_attn_fwd(ctypes.byref(big), P, P, P, P, P, 7, None, P, None, None) == -2


def test_schedule_static_rejects_bad_arguments():
    """The allocation-free schedule checks its arguments like
    sparse_attn_schedule and rejects problems whose counters exceed its 64 KiB
    device array ((chunks of 1024 tiles + 1) x 16 int32) before any HIP call."""
    lib = sa.library()
    ds = desc(B=2, H=3, N=1000)
    call = lambda d, *a: lib.sparse_attn_schedule_static(ctypes.byref(d), *a)
    assert call(ds, None, 7, P, None) == -1                          # null cnt
    assert call(ds, P, 7, None, None) == -1                          # null order
    assert call(ds, P, 0, P, None) == -1                             # kmax 0
    assert call(desc(block=96), P, 7, P, None) == -2                 # bad descriptor
    # 1023 chunks of 1024 tiles fit (1024 x 16 x 4 B = 64 KiB), 1024 do not
    fits = desc(B=1, H=1023, N=1024 * 64)
    assert lib.sparse_attn_workspace_size(ctypes.byref(fits), sa.SA_OP_SCHEDULE, 7) == 65536
    over = desc(B=1, H=1023, N=1024 * 64 + 64)
    assert lib.sparse_attn_workspace_size(ctypes.byref(over), sa.SA_OP_SCHEDULE, 7) > 65536
    assert call(over, P, 7, P, None) == -2

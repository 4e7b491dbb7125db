"""Python binding of libsparseattn (gfx950 block-sparse attention).

Argument marshalling only: every step of the computation runs in the HIP
kernels behind the C ABI declared in include/sparse_attn.h.  PyTorch provides
device memory (tensors, workspaces) and the current HIP stream.  There is no
fallback: if the shared library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

__all__ = [
    "LIB_PATH", "SparseAttnError", "SA_SELECT_ROW_TOPK", "SA_SELECT_HEAD_TOPK",
    "SA_OP_SELECT", "SA_OP_SCHEDULE", "SA_OP_SELECT_HEAD", "library", "sparse_attn_version",
    "sparse_attn_status_str", "sparse_attn_keep_count", "sparse_attn_workspace_size",
    "sparse_attn_num_tiles", "sparse_attn_select", "sparse_attn_schedule", "sparse_attn_fwd",
    "sparse_attn_schedule_static", "sparse_attn_quant_fp8", "sparse_attn_quant_fp8_tiles",
    "sparse_attn_fp8_tiles_bytes", "SA_FP8_K", "SA_FP8_V", "sparse_attn_fwd_fp8", "sparse_attn_comp_state",
    "sparse_attn_comp_out", "SA_OP_COMP_STATE", "COMP_RANK", "make_desc", "EXPORTED_SYMBOLS",
    "sparse_attn_quant_rows_fp8", "sparse_attn_linear_w8a8", "sparse_attn_bwd", "SA_OP_BWD",
]

# SPARSE_ATTN_LIB names another build of the same library (the CPU sanitizer
# build of the host layer that the argument-check tests run under); by
# default the in-tree gfx950 build is loaded.
LIB_PATH = os.environ.get("SPARSE_ATTN_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libsparseattn.so")

SA_SELECT_ROW_TOPK = 0
SA_SELECT_HEAD_TOPK = 1
SA_OP_SELECT, SA_OP_SCHEDULE, SA_OP_COMP_STATE, SA_OP_BWD, SA_OP_SELECT_HEAD = 0, 1, 2, 3, 4
COMP_RANK = 64

EXPORTED_SYMBOLS = (
    "sparse_attn_version", "sparse_attn_status_str", "sparse_attn_keep_count",
    "sparse_attn_workspace_size", "sparse_attn_num_tiles", "sparse_attn_select",
    "sparse_attn_schedule", "sparse_attn_fwd", "sparse_attn_quant_fp8",
    "sparse_attn_quant_fp8_tiles", "sparse_attn_fp8_tiles_bytes", "sparse_attn_fwd_fp8",
    "sparse_attn_comp_state", "sparse_attn_comp_out", "sparse_attn_quant_rows_fp8",
    "sparse_attn_linear_w8a8", "sparse_attn_bwd", "sparse_attn_schedule_static",
)


class SparseAttnError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {sparse_attn_status_str(status)} ({status})")
        self.status = status


class SparseAttnDesc(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("seqlen", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("block", ctypes.c_int32),
        ("q_stride", ctypes.c_int64 * 3), ("k_stride", ctypes.c_int64 * 3),
        ("v_stride", ctypes.c_int64 * 3), ("o_stride", ctypes.c_int64 * 3),
        ("softmax_scale", ctypes.c_float),
        ("causal_chunk", ctypes.c_int32), ("causal_window", ctypes.c_int32),
    ]


_LIB = None
_P = ctypes.c_void_p
_I32P = ctypes.POINTER(ctypes.c_int32)
_I64P = ctypes.POINTER(ctypes.c_int64)


def library() -> ctypes.CDLL:
    """The loaded shared library (raises if it has not been built)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        lib = ctypes.CDLL(LIB_PATH)
        D = ctypes.POINTER(SparseAttnDesc)
        sig = {
            "sparse_attn_version": (ctypes.c_int, []),
            "sparse_attn_status_str": (ctypes.c_char_p, [ctypes.c_int]),
            "sparse_attn_keep_count": (ctypes.c_int32, [ctypes.c_int32, ctypes.c_int32]),
            "sparse_attn_workspace_size": (ctypes.c_size_t, [D, ctypes.c_int32, ctypes.c_int32]),
            "sparse_attn_num_tiles": (ctypes.c_int64, [D]),
            "sparse_attn_select": (ctypes.c_int, [D, _P, _P, ctypes.c_int32, ctypes.c_int64,
                                                  _P, _P, ctypes.c_int32, _P, ctypes.c_size_t, _P]),
            "sparse_attn_schedule": (ctypes.c_int, [D, _P, ctypes.c_int32, _P, _P,
                                                    ctypes.c_size_t, _P]),
            "sparse_attn_schedule_static": (ctypes.c_int, [D, _P, ctypes.c_int32, _P, _P]),
            "sparse_attn_fwd": (ctypes.c_int, [D, _P, _P, _P, _P, _P, ctypes.c_int32, _P, _P, _P,
                                               _P]),
            "sparse_attn_quant_fp8": (ctypes.c_int, [D, _P, ctypes.POINTER(ctypes.c_int64),
                                                     _P, _P, _P]),
            "sparse_attn_quant_fp8_tiles": (ctypes.c_int, [D, _P, ctypes.POINTER(ctypes.c_int64),
                                                             ctypes.c_int32, _P, _P, _P]),
            "sparse_attn_fp8_tiles_bytes": (ctypes.c_int64, [D]),
            "sparse_attn_fwd_fp8": (ctypes.c_int, [D, _P, _P, _P, _P, _P, _P, _P, _P,
                                                   ctypes.c_int32, _P, _P, _P, _P]),
            "sparse_attn_comp_state": (ctypes.c_int, [D, ctypes.c_int32, _P, _I64P, _P, _P, _P,
                                                      _P, _P, ctypes.c_size_t, _P]),
            "sparse_attn_comp_out": (ctypes.c_int, [D, ctypes.c_int32, _P, _I64P, _P, _P, _P,
                                                    _P, ctypes.c_float, _P, _I64P, _P, _P, _P]),
            "sparse_attn_quant_rows_fp8": (ctypes.c_int, [_P, ctypes.c_int64, ctypes.c_int64,
                                                          ctypes.c_int64, _P, _P, _P]),
            "sparse_attn_bwd": (ctypes.c_int, [D, _P, _P, _P, _P, _P, _P, _P, _P,
                                               ctypes.c_int32, _P, _P, _P, _P, ctypes.c_size_t,
                                               _P]),
            "sparse_attn_linear_w8a8": (ctypes.c_int, [_P, _P, ctypes.c_int64, _P, _P,
                                                       ctypes.c_int64, _P, _P, ctypes.c_int64,
                                                       ctypes.c_int64, ctypes.c_int64,
                                                       ctypes.c_int64, _P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype, fn.argtypes = res, args
        _LIB = lib
    return _LIB


# ------------------------------------------------------------------ helpers
def _strides(t):
    if t is None:
        return (0, 0, 0)
    if t.dim() != 4 or t.stride(3) != 1:
        raise ValueError("expected a [B, H, N, d] tensor with contiguous channels")
    return tuple(t.stride()[:3])


def make_desc(q, k=None, v=None, o=None, block: int = 64, softmax_scale: float = 0.0,
              causal=None):
    """Descriptor for [B, H, N, d] tensors (strides in elements).  causal =
    (chunk_tokens, window_chunks) restricts attention to a causal window
    (window 0: every earlier chunk); None leaves it unrestricted."""
    B, H, N, d = q.shape
    desc = SparseAttnDesc()
    desc.batch, desc.heads, desc.seqlen, desc.head_dim, desc.block = B, H, N, d, block
    for field, t in (("q_stride", q), ("k_stride", k), ("v_stride", v), ("o_stride", o)):
        getattr(desc, field)[:] = _strides(t)
    desc.softmax_scale = softmax_scale
    if causal is not None:
        desc.causal_chunk, desc.causal_window = int(causal[0]), int(causal[1])
    return desc


def _stream(t):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _dense(t, name, dtype=torch.int32):
    """Index lists, counts and launch orders are dense C arrays at the ABI."""
    if t is not None and (not t.is_contiguous() or t.dtype != dtype):
        raise ValueError(f"{name} must be a contiguous {dtype} tensor")
    return t


def _check(status, what):
    if status != 0:
        raise SparseAttnError(status, what)


def _num_blocks(n, block):
    return -(-n // block)


# --------------------------------------------------------------------- API
def sparse_attn_version() -> int:
    return library().sparse_attn_version()


def sparse_attn_status_str(status: int) -> str:
    return library().sparse_attn_status_str(status).decode()


def sparse_attn_keep_count(keep_bp: int, nkb: int) -> int:
    return library().sparse_attn_keep_count(keep_bp, nkb)


def sparse_attn_workspace_size(desc: SparseAttnDesc, op: int, kmax: int = 1) -> int:
    return library().sparse_attn_workspace_size(ctypes.byref(desc), op, kmax)


def sparse_attn_num_tiles(desc: SparseAttnDesc) -> int:
    return library().sparse_attn_num_tiles(ctypes.byref(desc))


def _workspace(desc, op, kmax, device):
    n = sparse_attn_workspace_size(desc, op, kmax)
    if n == 0:
        raise SparseAttnError(-2, "workspace size")
    return torch.empty(n, dtype=torch.uint8, device=device)


def sparse_attn_select(q, k, budget: int, block: int = 64, mode: int = SA_SELECT_ROW_TOPK,
                       kmax: int | None = None, idx=None, cnt=None, ws=None, causal=None):
    """Block selection on bf16 q, k [B, H, N, 128].  Returns (idx, cnt):
    idx int32 [B, H, nb, kmax] (ascending, -1 padded), cnt int32 [B, H, nb]."""
    B, H, N, _ = q.shape
    nb = _num_blocks(N, block)
    if kmax is None:
        kmax = budget if mode == SA_SELECT_ROW_TOPK else nb
    desc = make_desc(q, k, block=block, causal=causal)
    if idx is None:
        idx = torch.empty(B, H, nb, kmax, dtype=torch.int32, device=q.device)
    if cnt is None:
        cnt = torch.empty(B, H, nb, dtype=torch.int32, device=q.device)
    _dense(idx, "idx"), _dense(cnt, "cnt")
    if ws is None:
        op = SA_OP_SELECT if mode == SA_SELECT_ROW_TOPK else SA_OP_SELECT_HEAD
        ws = _workspace(desc, op, kmax, q.device)
    st = library().sparse_attn_select(ctypes.byref(desc), _ptr(q), _ptr(k), mode, budget,
                                      _ptr(idx), _ptr(cnt), kmax, _ptr(ws), ws.numel(),
                                      _stream(q))
    _check(st, "sparse_attn_select")
    return idx, cnt


def sparse_attn_schedule(cnt, seqlen: int, kmax: int, block: int = 64, order=None, ws=None):
    """Launch order of the 64-row query tiles for the lists' lengths ``cnt``
    [B, H, nb].  Returns int32 [B * H * ceil(seqlen / 64)]."""
    B, H, _ = cnt.shape
    _dense(cnt, "cnt")
    _dense(order, "order")
    desc = SparseAttnDesc()
    desc.batch, desc.heads, desc.seqlen, desc.head_dim, desc.block = B, H, seqlen, 128, block
    n = sparse_attn_num_tiles(desc)
    if n < 0:
        raise SparseAttnError(-2, "sparse_attn_num_tiles")
    if order is None:
        order = torch.empty(n, dtype=torch.int32, device=cnt.device)
    if ws is None:
        ws = _workspace(desc, SA_OP_SCHEDULE, kmax, cnt.device)
    st = library().sparse_attn_schedule(ctypes.byref(desc), _ptr(cnt), kmax, _ptr(order),
                                        _ptr(ws), ws.numel(), _stream(cnt))
    _check(st, "sparse_attn_schedule")
    return order


def sparse_attn_schedule_static(cnt, seqlen: int, kmax: int, order, block: int = 64):
    """sparse_attn_schedule without a workspace (the library's per-GPU device
    array holds the counters): writes the launch order into the caller's
    ``order`` (int32 [B * H * ceil(seqlen / 64)]) and allocates nothing."""
    B, H, _ = cnt.shape
    _dense(cnt, "cnt")
    _dense(order, "order")
    desc = SparseAttnDesc()
    desc.batch, desc.heads, desc.seqlen, desc.head_dim, desc.block = B, H, seqlen, 128, block
    if order.numel() != sparse_attn_num_tiles(desc):
        raise ValueError("order must hold one int32 per query tile")
    st = library().sparse_attn_schedule_static(ctypes.byref(desc), _ptr(cnt), kmax, _ptr(order),
                                               _stream(cnt))
    _check(st, "sparse_attn_schedule_static")
    return order


def sparse_attn_fwd(q, k, v, idx, cnt, block: int = 64, softmax_scale: float = 0.0,
                    with_lse: bool = True, order=None, o=None, lse=None, causal=None):
    """Block-sparse attention forward on bf16 q, k, v [B, H, N, 128] with the
    lists from sparse_attn_select (and optionally the launch order from
    sparse_attn_schedule).  Returns (o bf16 [B, H, N, 128], lse fp32
    [B, H, N] or None)."""
    B, H, N, _ = q.shape
    kmax = idx.shape[-1]
    _dense(idx, "idx"), _dense(cnt, "cnt"), _dense(order, "order")
    if o is None:
        o = torch.empty_like(q, memory_format=torch.contiguous_format)
    if with_lse and lse is None:
        lse = torch.empty(B, H, N, dtype=torch.float32, device=q.device)
    desc = make_desc(q, k, v, o, block=block, softmax_scale=softmax_scale, causal=causal)
    st = library().sparse_attn_fwd(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(idx),
                                   _ptr(cnt), kmax, _ptr(order), _ptr(o),
                                   _ptr(lse if with_lse else None), _stream(q))
    _check(st, "sparse_attn_fwd")
    return o, (lse if with_lse else None)


def sparse_attn_quant_fp8(x, block: int = 64, x8=None, scale=None):
    """e4m3 quantisation with one power-of-two scale per block of tokens.
    Returns (x8 uint8 [B, H, N, 128] contiguous, scale fp32 [B, H, nb])."""
    B, H, N, _ = x.shape
    desc = make_desc(x, block=block)
    if x8 is None:
        x8 = torch.empty(B, H, N, x.shape[3], dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty(B, H, _num_blocks(N, block), dtype=torch.float32, device=x.device)
    xs = (ctypes.c_int64 * 3)(*_strides(x))
    st = library().sparse_attn_quant_fp8(ctypes.byref(desc), _ptr(x), xs, _ptr(x8),
                                         _ptr(scale), _stream(x))
    _check(st, "sparse_attn_quant_fp8")
    return x8, scale


SA_FP8_K, SA_FP8_V = 0, 1


def sparse_attn_quant_fp8_tiles(x, operand: int, block: int = 64, x8=None, scale=None):
    """The quantisation of sparse_attn_quant_fp8 with the codes in the fp8
    forward's K (SA_FP8_K) or V (SA_FP8_V) operand order.  Returns (x8 uint8
    [B, H, ceil(N / 64), 8192], scale fp32 [B, H, nb])."""
    B, H, N, _ = x.shape
    desc = make_desc(x, block=block)
    if x8 is None:
        x8 = torch.empty(B, H, -(-N // 64), 8192, dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty(B, H, _num_blocks(N, block), dtype=torch.float32, device=x.device)
    _dense(x8, "x8", torch.uint8)
    if x8.numel() < library().sparse_attn_fp8_tiles_bytes(ctypes.byref(desc)):
        raise ValueError("x8 is smaller than sparse_attn_fp8_tiles_bytes")
    xs = (ctypes.c_int64 * 3)(*_strides(x))
    st = library().sparse_attn_quant_fp8_tiles(ctypes.byref(desc), _ptr(x), xs, operand,
                                               _ptr(x8), _ptr(scale), _stream(x))
    _check(st, "sparse_attn_quant_fp8_tiles")
    return x8, scale


def sparse_attn_fwd_fp8(q8, sq, k8, sk, v8, sv, idx, cnt, block: int = 64,
                        softmax_scale: float = 0.0, with_lse: bool = True, order=None, o=None,
                        lse=None, causal=None):
    """Block-sparse attention forward on e4m3 operands: q8 from
    sparse_attn_quant_fp8, k8 and v8 from sparse_attn_quant_fp8_tiles
    (SA_FP8_K, SA_FP8_V).  Returns (o bf16 [B, H, N, 128], lse or None)."""
    B, H, N, d = q8.shape
    kmax = idx.shape[-1]
    _dense(idx, "idx"), _dense(cnt, "cnt"), _dense(order, "order")
    for name, t in (("q8", q8), ("k8", k8), ("v8", v8)):
        _dense(t, name, torch.uint8)
    for name, t in (("sq", sq), ("sk", sk), ("sv", sv)):
        _dense(t, name, torch.float32)
    if o is None:
        o = torch.empty(B, H, N, d, dtype=torch.bfloat16, device=q8.device)
    if with_lse and lse is None:
        lse = torch.empty(B, H, N, dtype=torch.float32, device=q8.device)
    desc = make_desc(o, o=o, block=block, softmax_scale=softmax_scale, causal=causal)
    st = library().sparse_attn_fwd_fp8(ctypes.byref(desc), _ptr(q8), _ptr(sq), _ptr(k8),
                                       _ptr(sk), _ptr(v8), _ptr(sv), _ptr(idx), _ptr(cnt), kmax,
                                       _ptr(order), _ptr(o), _ptr(lse if with_lse else None),
                                       _stream(q8))
    _check(st, "sparse_attn_fwd_fp8")
    return o, (lse if with_lse else None)


def default_softmax_scale(d: int) -> float:
    """fp32(1/sqrt(d)), the scale the library uses when 0 is passed."""
    return float(torch.tensor(1.0 / math.sqrt(d), dtype=torch.float32))


def _st3(strides):
    return (ctypes.c_int64 * 3)(*strides)


def sparse_attn_comp_state(k_norm, v, pk, rope, state=None, ws=None, causal=None):
    """Low-rank state C = sum_j k~_j v_j^T of the compensation branch.
    k_norm, v bf16 [B, H, N, 128]; pk bf16 [H, 64, 128]; rope fp32 [N, 32, 2].
    Returns the state transposed, fp32 [B, H, 128, 64] (state[..., c, m] =
    C[m, c]); under a causal window (chunk, window) one state per chunk,
    [B, H, ceil(N / chunk), 128, 64]."""
    B, H, N, d = k_norm.shape
    desc = make_desc(k_norm, k_norm, v, causal=causal)
    if state is None:
        if causal is None or int(causal[0]) <= 0:
            shape = (B, H, d, COMP_RANK)
        else:
            shape = (B, H, -(-N // min(int(causal[0]), N)), d, COMP_RANK)
        state = torch.empty(shape, dtype=torch.float32, device=k_norm.device)
    for t, name, dt in ((pk, "pk", torch.bfloat16), (rope, "rope", torch.float32),
                        (state, "state", torch.float32)):
        _dense(t, name, dt)
    if ws is None:
        ws = _workspace(desc, SA_OP_COMP_STATE, 1, k_norm.device)
    st = library().sparse_attn_comp_state(ctypes.byref(desc), COMP_RANK, _ptr(k_norm),
                                          _st3(_strides(k_norm)), _ptr(v), _ptr(pk), _ptr(rope),
                                          _ptr(state), _ptr(ws), ws.numel(), _stream(k_norm))
    _check(st, "sparse_attn_comp_state")
    return state


def sparse_attn_comp_out(q_norm, pq, rope, state, gate, o_s, gamma=None, eps: float = 1e-6,
                         o=None, causal=None):
    """Gated output O = O_s + g * rms(O_s) * RMSNorm(q~^T C) (o may be o_s).
    gate fp32 [B, H, N] (any strides, including 0); gamma fp32 [H, 128] or None;
    causal (chunk, window) as for the state."""
    B, H, N, d = q_norm.shape
    if o is None:
        o = torch.empty_like(o_s)
    if _strides(o) != _strides(o_s):
        raise ValueError("o and o_s must share their strides")
    desc = make_desc(q_norm, o=o_s, causal=causal)
    for t, name, dt in ((pq, "pq", torch.bfloat16), (rope, "rope", torch.float32),
                        (state, "state", torch.float32), (gamma, "gamma", torch.float32)):
        _dense(t, name, dt)
    if gate.dtype != torch.float32 or gate.dim() != 3:
        raise ValueError("gate must be a float32 [B, H, N] tensor")
    st = library().sparse_attn_comp_out(ctypes.byref(desc), COMP_RANK, _ptr(q_norm),
                                        _st3(_strides(q_norm)), _ptr(pq), _ptr(rope),
                                        _ptr(state), _ptr(gamma), eps, _ptr(gate),
                                        _st3(gate.stride()), _ptr(o_s), _ptr(o), _stream(q_norm))
    _check(st, "sparse_attn_comp_out")
    return o


# ------------------------------------------------------- W8A8 fp8 linear layers
def _rows_2d(t, name, dtype):
    if t.dim() != 2 or t.dtype != dtype or t.stride(1) != 1:
        raise ValueError(f"{name} must be a 2-D {dtype} tensor with unit column stride")


def sparse_attn_quant_rows_fp8(x, q=None, scale=None):
    """Per-row e4m3 quantisation of bf16 x [rows, cols] (any row stride).
    Returns (q uint8 [rows, cols] contiguous, scale fp32 [rows])."""
    _rows_2d(x, "x", torch.bfloat16)
    rows, cols = x.shape
    if q is None:
        q = torch.empty(rows, cols, dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty(rows, dtype=torch.float32, device=x.device)
    if not q.is_contiguous() or tuple(q.shape) != (rows, cols) or q.dtype != torch.uint8:
        raise ValueError("q must be a contiguous uint8 [rows, cols] tensor")
    _dense(scale, "scale", torch.float32)
    st = library().sparse_attn_quant_rows_fp8(_ptr(x), rows, cols, x.stride(0), _ptr(q),
                                              _ptr(scale), _stream(x))
    _check(st, "sparse_attn_quant_rows_fp8")
    return q, scale


def sparse_attn_linear_w8a8(xq, sx, wq, sw, bias=None, y=None):
    """y [M, N] bf16 = (xq wq^T) * sx sw^T + bias over e4m3 codes xq [M, K],
    wq [N, K] (unit column stride, any row stride) and fp32 scales sx [M],
    sw [N]; bias fp32 [N] or None."""
    _rows_2d(xq, "xq", torch.uint8)
    _rows_2d(wq, "wq", torch.uint8)
    M, K = xq.shape
    N = wq.shape[0]
    if wq.shape[1] != K:
        raise ValueError("xq and wq must have the same K")
    _dense(sx, "sx", torch.float32)
    _dense(sw, "sw", torch.float32)
    if bias is not None:
        _dense(bias, "bias", torch.float32)
    if y is None:
        y = torch.empty(M, N, dtype=torch.bfloat16, device=xq.device)
    _rows_2d(y, "y", torch.bfloat16)
    st = library().sparse_attn_linear_w8a8(
        _ptr(xq), _ptr(sx), xq.stride(0), _ptr(wq), _ptr(sw), wq.stride(0),
        None if bias is None else _ptr(bias), _ptr(y), y.stride(0), M, N, K, _stream(xq))
    _check(st, "sparse_attn_linear_w8a8")
    return y


# ---------------------------------------------------------------- backward
def sparse_attn_bwd(q, k, v, o, d_o, lse, idx, cnt, block: int = 64,
                    softmax_scale: float = 0.0, dq=None, dk=None, dv=None, ws=None,
                    causal=None):
    """Gradients (dq, dk, dv) bf16 of the sparse forward for upstream d_o
    (laid out like o), given the forward's lists, output and lse (and its
    causal window (chunk, window), if any)."""
    kmax = idx.shape[-1]
    _dense(idx, "idx"), _dense(cnt, "cnt"), _dense(lse, "lse", torch.float32)
    if tuple(d_o.stride()) != tuple(o.stride()):
        raise ValueError("d_o must be laid out like o")
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(k) if dk is None else dk
    dv = torch.empty_like(v) if dv is None else dv
    for name, a, ref in (("dq", dq, q), ("dk", dk, k), ("dv", dv, v)):
        if tuple(a.stride()) != tuple(ref.stride()):
            raise ValueError(f"{name} must be laid out like its input")
    desc = make_desc(q, k, v, o, block=block, softmax_scale=softmax_scale, causal=causal)
    if ws is None:
        ws = _workspace(desc, SA_OP_BWD, kmax, q.device)
    st = library().sparse_attn_bwd(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                   _ptr(d_o), _ptr(lse), _ptr(idx), _ptr(cnt), kmax, _ptr(dq),
                                   _ptr(dk), _ptr(dv), _ptr(ws), ws.numel(), _stream(q))
    _check(st, "sparse_attn_bwd")
    return dq, dk, dv

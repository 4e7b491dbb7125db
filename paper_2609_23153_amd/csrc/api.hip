// C ABI of the library: argument checks on the host, then launches.
// Every check runs before the first HIP call, so invalid calls launch nothing
// (and can be exercised on a machine without a GPU).
#include <math.h>

#include "launch.h"
#include "sparse_attn.h"

namespace {

using sa::Shape;
using sa::Strides;

constexpr int kMaxBlocks = 4096;  // nb limit of the selection kernels

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool strides_ok(const int64_t st[3]) {
  for (int i = 0; i < 3; ++i)
    if (st[i] < 0 || (st[i] & 7) != 0) return false;
  return true;
}

// Shape checks shared by every call.  Returns SA_OK or an error code.
int check_desc(const sparse_attn_desc* d, Shape* s) {
  if (!d) return SA_ERR_INVALID_ARG;
  if (d->batch < 1 || d->heads < 1 || d->seqlen < 1) return SA_ERR_INVALID_ARG;
  if (!(d->softmax_scale >= 0.f) || isinf(d->softmax_scale)) return SA_ERR_INVALID_ARG;
  if (d->head_dim != 128) return SA_ERR_UNSUPPORTED;
  if (d->block != 64 && d->block != 128) return SA_ERR_UNSUPPORTED;
  const int64_t nb = (d->seqlen + (int64_t)d->block - 1) / d->block;
  if (nb > kMaxBlocks) return SA_ERR_UNSUPPORTED;
  // query tiles (and so launch slots) must fit the 32-bit tile index
  const int64_t ntiles = (d->seqlen + 63) / 64;
  if ((int64_t)d->batch * d->heads * ntiles > (int64_t)1 << 30) return SA_ERR_UNSUPPORTED;
  // causal window: chunk >= 0 tokens (0: none), window >= 0 chunks (0: all
  // earlier chunks), and no window without chunks
  if (d->causal_chunk < 0 || d->causal_window < 0) return SA_ERR_INVALID_ARG;
  if (d->causal_chunk == 0 && d->causal_window != 0) return SA_ERR_INVALID_ARG;
  s->causal_chunk = d->causal_chunk;
  s->causal_window = d->causal_window;
  s->B = d->batch;
  s->H = d->heads;
  s->N = d->seqlen;
  s->block = d->block;
  s->nb = (int)nb;
  return SA_OK;
}

Strides to_strides(const int64_t st[3]) { return Strides{st[0], st[1], st[2]}; }

// The kernels address one head's rows with 32-bit byte offsets, up to the
// last row of the last (padded) 64-token tile.
bool offsets_fit(const Shape& s, const int64_t st[3], int elem_bytes) {
  return ((int64_t)s.N + 64) * st[2] * elem_bytes + 256 < ((int64_t)1 << 32);
}

float effective_scale(const sparse_attn_desc* d) {
  return d->softmax_scale > 0.f ? d->softmax_scale : (float)(1.0 / sqrt((double)d->head_dim));
}

int launch_status(hipError_t e) { return e == hipSuccess ? SA_OK : SA_ERR_LAUNCH; }

int check_lists(const Shape& s, const int32_t* idx, const int32_t* cnt, int32_t kmax) {
  if (!idx || !cnt) return SA_ERR_INVALID_ARG;
  if (kmax < 1 || kmax > (1 << 16)) return SA_ERR_INVALID_ARG;
  return SA_OK;
}

}  // namespace

extern "C" {

int sparse_attn_version(void) { return SPARSE_ATTN_VERSION; }

const char* sparse_attn_status_str(int status) {
  switch (status) {
    case SA_OK: return "ok";
    case SA_ERR_INVALID_ARG: return "invalid argument";
    case SA_ERR_UNSUPPORTED: return "unsupported problem shape";
    case SA_ERR_WORKSPACE: return "workspace too small";
    case SA_ERR_LAUNCH: return "HIP launch failed";
    case SA_ERR_DEVICE: return "no usable gfx950 device";
    default: return "unknown status";
  }
}

int32_t sparse_attn_keep_count(int32_t keep_bp, int32_t nkb) {
  if (keep_bp < 1 || nkb < 1) return -1;
  const int64_t k = ((int64_t)keep_bp * nkb + 9999) / 10000;
  return (int32_t)(k < 1 ? 1 : (k > nkb ? nkb : k));
}

size_t sparse_attn_workspace_size(const sparse_attn_desc* desc, int32_t op, int32_t kmax) {
  Shape s;
  if (check_desc(desc, &s) != SA_OK) return 0;
  switch (op) {
    case SA_OP_SELECT: return sa::select_workspace_bytes(s);
    case SA_OP_SELECT_HEAD: return sa::select_head_workspace_bytes(s);
    case SA_OP_SCHEDULE: return kmax >= 1 ? sa::schedule_workspace_bytes(s) : 0;
    case SA_OP_COMP_STATE: return sa::comp_state_workspace_bytes(s);
    case SA_OP_BWD: return sa::bwd_workspace_bytes(s);
    default: return 0;
  }
}

int64_t sparse_attn_num_tiles(const sparse_attn_desc* desc) {
  Shape s;
  if (check_desc(desc, &s) != SA_OK) return -1;
  return sa::num_query_tiles(s);
}

int sparse_attn_schedule(const sparse_attn_desc* desc, const int32_t* cnt, int32_t kmax,
                         int32_t* order, void* ws, size_t ws_bytes, void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (!order || !ws) return SA_ERR_INVALID_ARG;
  if ((st = check_lists(s, cnt, cnt, kmax)) != SA_OK) return st;
  if (ws_bytes < sa::schedule_workspace_bytes(s)) return SA_ERR_WORKSPACE;
  return launch_status(
      sa::launch_schedule(s, cnt, kmax, order, ws, static_cast<hipStream_t>(stream)));
}

int sparse_attn_schedule_static(const sparse_attn_desc* desc, const int32_t* cnt, int32_t kmax,
                                int32_t* order, void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (!order) return SA_ERR_INVALID_ARG;
  if ((st = check_lists(s, cnt, cnt, kmax)) != SA_OK) return st;
  if (sa::schedule_workspace_bytes(s) > sa::kStaticScheduleScratchBytes) return SA_ERR_UNSUPPORTED;
  int32_t* scratch = nullptr;
  if (sa::static_schedule_scratch(&scratch) != hipSuccess) return SA_ERR_DEVICE;
  return launch_status(
      sa::launch_schedule(s, cnt, kmax, order, scratch, static_cast<hipStream_t>(stream)));
}

int sparse_attn_select(const sparse_attn_desc* desc, const void* q, const void* k, int32_t mode,
                       int64_t budget, int32_t* idx, int32_t* cnt, int32_t kmax, void* ws,
                       size_t ws_bytes, void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (!q || !k || !idx || !cnt || !ws) return SA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !strides_ok(desc->q_stride) || !strides_ok(desc->k_stride))
    return SA_ERR_INVALID_ARG;
  if (kmax < 1) return SA_ERR_INVALID_ARG;
  if (mode == SA_SELECT_ROW_TOPK) {
    if (budget < 1 || budget > s.nb || kmax < budget) return SA_ERR_INVALID_ARG;
  } else if (mode == SA_SELECT_HEAD_TOPK) {
    if (budget < s.nb || budget > (int64_t)s.nb * s.nb) return SA_ERR_INVALID_ARG;
    if (s.causal_chunk > 0) return SA_ERR_UNSUPPORTED;  // whole-head budget: no causal window
  } else {
    return SA_ERR_INVALID_ARG;
  }
  if (ws_bytes < (mode == SA_SELECT_ROW_TOPK ? sa::select_workspace_bytes(s)
                                              : sa::select_head_workspace_bytes(s)))
    return SA_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  if (mode == SA_SELECT_ROW_TOPK)
    return launch_status(sa::launch_select_row(s, q, to_strides(desc->q_stride), k,
                                               to_strides(desc->k_stride), (int)budget, kmax,
                                               idx, cnt, ws, hs));
  const hipError_t e = sa::launch_select_head(s, q, to_strides(desc->q_stride), k,
                                              to_strides(desc->k_stride), budget, kmax, idx,
                                              cnt, ws, hs);
  return e == hipErrorNotSupported ? SA_ERR_UNSUPPORTED : launch_status(e);
}

int sparse_attn_fwd(const sparse_attn_desc* desc, const void* q, const void* k, const void* v,
                    const int32_t* idx, const int32_t* cnt, int32_t kmax, const int32_t* order,
                    void* o, float* lse, void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (!q || !k || !v || !o) return SA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return SA_ERR_INVALID_ARG;
  if (!strides_ok(desc->q_stride) || !strides_ok(desc->k_stride) ||
      !strides_ok(desc->v_stride) || !strides_ok(desc->o_stride))
    return SA_ERR_INVALID_ARG;
  if ((st = check_lists(s, idx, cnt, kmax)) != SA_OK) return st;
  if (!offsets_fit(s, desc->q_stride, 2) || !offsets_fit(s, desc->k_stride, 2) ||
      !offsets_fit(s, desc->v_stride, 2))
    return SA_ERR_UNSUPPORTED;
  sa::FwdArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.lse = lse;
  a.qs = to_strides(desc->q_stride);
  a.ks = to_strides(desc->k_stride);
  a.vs = to_strides(desc->v_stride);
  a.os = to_strides(desc->o_stride);
  a.idx = idx;
  a.cnt = cnt;
  a.order = order;
  a.kmax = kmax;
  a.softmax_scale = effective_scale(desc);
  return launch_status(sa::launch_fwd_bf16(s, a, static_cast<hipStream_t>(stream)));
}

int sparse_attn_quant_fp8(const sparse_attn_desc* desc, const void* x, const int64_t x_stride[3],
                          uint8_t* x8, float* scale, void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (!x || !x_stride || !x8 || !scale) return SA_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(x8) || !strides_ok(x_stride)) return SA_ERR_INVALID_ARG;
  return launch_status(
      sa::launch_quant_fp8(s, x, to_strides(x_stride), x8, scale, static_cast<hipStream_t>(stream)));
}

int sparse_attn_quant_fp8_tiles(const sparse_attn_desc* desc, const void* x,
                                const int64_t x_stride[3], int32_t operand, uint8_t* x8,
                                float* scale, void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (!x || !x_stride || !x8 || !scale) return SA_ERR_INVALID_ARG;
  if (operand != SA_FP8_K && operand != SA_FP8_V) return SA_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(x8) || !strides_ok(x_stride)) return SA_ERR_INVALID_ARG;
  return launch_status(sa::launch_quant_fp8_tiles(s, x, to_strides(x_stride), operand == SA_FP8_V,
                                                  x8, scale, static_cast<hipStream_t>(stream)));
}

int64_t sparse_attn_fp8_tiles_bytes(const sparse_attn_desc* desc) {
  Shape s;
  if (check_desc(desc, &s) != SA_OK) return -1;
  return (int64_t)s.B * s.H * ((s.N + 63) / 64) * 8192;
}

int sparse_attn_fwd_fp8(const sparse_attn_desc* desc, const uint8_t* q8, const float* sq,
                        const uint8_t* k8, const float* sk, const uint8_t* v8, const float* sv,
                        const int32_t* idx, const int32_t* cnt, int32_t kmax,
                        const int32_t* order, void* o, float* lse, void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (!q8 || !sq || !k8 || !sk || !v8 || !sv || !o) return SA_ERR_INVALID_ARG;
  if (!aligned16(q8) || !aligned16(k8) || !aligned16(v8) || !aligned16(o))
    return SA_ERR_INVALID_ARG;
  if (!strides_ok(desc->o_stride)) return SA_ERR_INVALID_ARG;
  if ((st = check_lists(s, idx, cnt, kmax)) != SA_OK) return st;
  const int64_t tok = 128, head = (int64_t)s.N * tok, bat = head * s.H;
  sa::FwdArgs a{};
  a.q = q8;
  a.k = k8;
  a.v = v8;
  a.o = o;
  a.lse = lse;
  a.qs = a.ks = a.vs = Strides{bat, head, tok};
  a.os = to_strides(desc->o_stride);
  a.idx = idx;
  a.cnt = cnt;
  a.sq = sq;
  a.sk = sk;
  a.sv = sv;
  a.order = order;
  a.kmax = kmax;
  a.softmax_scale = effective_scale(desc);
  return launch_status(sa::launch_fwd_fp8(s, a, static_cast<hipStream_t>(stream)));
}

int sparse_attn_quant_rows_fp8(const void* x, int64_t rows, int64_t cols, int64_t ldx, uint8_t* q,
                               float* scale, void* stream) {
  if (!x || !q || !scale) return SA_ERR_INVALID_ARG;
  if (rows < 0 || cols < 8 || (cols & 7) != 0 || ldx < cols || (ldx & 7) != 0)
    return SA_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(q)) return SA_ERR_INVALID_ARG;
  if (cols > ((int64_t)1 << 30) || rows > ((int64_t)1 << 40)) return SA_ERR_UNSUPPORTED;
  return launch_status(sa::launch_quant_rows_fp8(x, ldx, rows, (int)cols, q, scale,
                                                 static_cast<hipStream_t>(stream)));
}

int sparse_attn_linear_w8a8(const uint8_t* xq, const float* sx, int64_t ldx, const uint8_t* wq,
                            const float* sw, int64_t ldw, const float* bias, void* y, int64_t ldy,
                            int64_t M, int64_t N, int64_t K, void* stream) {
  if (!xq || !sx || !wq || !sw || !y) return SA_ERR_INVALID_ARG;
  if (M < 0 || N < 0 || K < 256 || (K & 127) != 0 || (N & 7) != 0) return SA_ERR_INVALID_ARG;
  if (ldx < K || (ldx & 15) != 0 || ldw < K || (ldw & 15) != 0 || ldy < N || (ldy & 7) != 0)
    return SA_ERR_INVALID_ARG;
  if (!aligned16(xq) || !aligned16(wq) || !aligned16(sw) || (bias && !aligned16(bias)) ||
      !aligned16(y))
    return SA_ERR_INVALID_ARG;
  // 32-bit tile counts and per-tile byte offsets of the kernel
  if (M >= ((int64_t)1 << 31) || N >= ((int64_t)1 << 31) || K >= ((int64_t)1 << 31))
    return SA_ERR_UNSUPPORTED;
  if (256 * ldx >= ((int64_t)1 << 32) || 256 * ldw >= ((int64_t)1 << 32)) return SA_ERR_UNSUPPORTED;
  if (((M + 255) / 256) * ((N + 255) / 256) >= ((int64_t)1 << 31)) return SA_ERR_UNSUPPORTED;
  sa::LinearIn in{};
  in.xq = xq;
  in.sx = sx;
  in.wq = wq;
  in.sw = sw;
  in.bias = bias;
  in.y = y;
  in.ldx = ldx;
  in.ldw = ldw;
  in.ldy = ldy;
  in.M = M;
  in.N = N;
  in.K = K;
  in.group_m = 0;
  return launch_status(sa::launch_linear_w8a8(in, static_cast<hipStream_t>(stream)));
}

int sparse_attn_bwd(const sparse_attn_desc* desc, const void* q, const void* k, const void* v,
                    const void* o, const void* d_o, const float* lse, const int32_t* idx,
                    const int32_t* cnt, int32_t kmax, void* dq, void* dk, void* dv, void* ws,
                    size_t ws_bytes, void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (!q || !k || !v || !o || !d_o || !lse || !dq || !dk || !dv || !ws) return SA_ERR_INVALID_ARG;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(d_o) ||
      !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
    return SA_ERR_INVALID_ARG;
  if (!strides_ok(desc->q_stride) || !strides_ok(desc->k_stride) ||
      !strides_ok(desc->v_stride) || !strides_ok(desc->o_stride))
    return SA_ERR_INVALID_ARG;
  if ((st = check_lists(s, idx, cnt, kmax)) != SA_OK) return st;
  // the backward kernels address q, k, v, o and d_o rows of one head with
  // 32-bit byte offsets, as the forward does
  if (!offsets_fit(s, desc->q_stride, 2) || !offsets_fit(s, desc->k_stride, 2) ||
      !offsets_fit(s, desc->v_stride, 2) || !offsets_fit(s, desc->o_stride, 2))
    return SA_ERR_UNSUPPORTED;
  if (ws_bytes < sa::bwd_workspace_bytes(s)) return SA_ERR_WORKSPACE;
  sa::BwdIn in{};
  in.q = q;
  in.k = k;
  in.v = v;
  in.o = o;
  in.dout = d_o;
  in.lse = lse;
  in.idx = idx;
  in.cnt = cnt;
  in.dq = dq;
  in.dk = dk;
  in.dv = dv;
  in.qs = to_strides(desc->q_stride);
  in.ks = to_strides(desc->k_stride);
  in.vs = to_strides(desc->v_stride);
  in.os = to_strides(desc->o_stride);
  in.kmax = kmax;
  in.softmax_scale = effective_scale(desc);
  return launch_status(sa::launch_bwd(s, in, ws, static_cast<hipStream_t>(stream)));
}

}  // extern "C"

// ---- compensation branch (paper §2 Eq. comp-sparse, §4.1) -----------------
namespace {
// Strides of a [B][H][N] fp32 gate: non-negative (0 broadcasts).
bool gate_strides_ok(const int64_t st[3]) {
  return st && st[0] >= 0 && st[1] >= 0 && st[2] >= 0;
}
}  // namespace

int sparse_attn_comp_state(const sparse_attn_desc* desc, int32_t rank, const void* k_norm,
                           const int64_t kn_stride[3], const void* v, const void* pk,
                           const float* rope, float* state, void* ws, size_t ws_bytes,
                           void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (rank != 64) return SA_ERR_UNSUPPORTED;
  if (!k_norm || !kn_stride || !v || !pk || !rope || !state || !ws) return SA_ERR_INVALID_ARG;
  if (!aligned16(k_norm) || !aligned16(v) || !aligned16(pk) || !aligned16(rope) ||
      !aligned16(state))
    return SA_ERR_INVALID_ARG;
  if (!strides_ok(kn_stride) || !strides_ok(desc->v_stride)) return SA_ERR_INVALID_ARG;
  if (!offsets_fit(s, kn_stride, 2) || !offsets_fit(s, desc->v_stride, 2)) return SA_ERR_UNSUPPORTED;
  if ((int64_t)s.N * 256 >= ((int64_t)1 << 32)) return SA_ERR_UNSUPPORTED;  // rope offsets
  if (ws_bytes < sa::comp_state_workspace_bytes(s)) return SA_ERR_WORKSPACE;
  sa::CompStateIn in{};
  in.k_norm = k_norm;
  in.v = v;
  in.pk = pk;
  in.rope = rope;
  in.kns = to_strides(kn_stride);
  in.vs = to_strides(desc->v_stride);
  return launch_status(
      sa::launch_comp_state(s, in, state, ws, static_cast<hipStream_t>(stream)));
}

int sparse_attn_comp_out(const sparse_attn_desc* desc, int32_t rank, const void* q_norm,
                         const int64_t qn_stride[3], const void* pq, const float* rope,
                         const float* state, const float* gamma, float eps, const float* gate,
                         const int64_t gate_stride[3], const void* o_s, void* o,
                         void* stream) {
  Shape s;
  int st = check_desc(desc, &s);
  if (st != SA_OK) return st;
  if (rank != 64) return SA_ERR_UNSUPPORTED;
  if (!q_norm || !qn_stride || !pq || !rope || !state || !gate || !o_s || !o)
    return SA_ERR_INVALID_ARG;
  if (!aligned16(q_norm) || !aligned16(pq) || !aligned16(rope) || !aligned16(state) ||
      !aligned16(o_s) || !aligned16(o) || (gamma && !aligned16(gamma)))
    return SA_ERR_INVALID_ARG;
  if (!strides_ok(qn_stride) || !strides_ok(desc->o_stride) || !gate_strides_ok(gate_stride))
    return SA_ERR_INVALID_ARG;
  if (!(eps >= 0.f) || isinf(eps)) return SA_ERR_INVALID_ARG;
  sa::CompOutIn in{};
  in.q_norm = q_norm;
  in.pq = pq;
  in.rope = rope;
  in.state = state;
  in.gamma = gamma;
  in.gate = gate;
  in.o_s = o_s;
  in.o = o;
  in.qns = to_strides(qn_stride);
  in.gs = to_strides(gate_stride);
  in.oss = to_strides(desc->o_stride);
  in.eps = eps;
  return launch_status(sa::launch_comp_out(s, in, static_cast<hipStream_t>(stream)));
}

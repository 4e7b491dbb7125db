/*
 * sparse_attn.h -- C ABI of the MI355X (gfx950) block-sparse attention library.
 *
 * The library computes the sparse branch O_s = A_M(Q, K, V) of compensated
 * sparse attention (paper §2, Eq. comp-sparse; §4.1): the attention matrix is
 * cut into contiguous query and key blocks (§2 "Block sparsity"), a selector
 * M_phi keeps a few key blocks per query block, and exact softmax attention is
 * evaluated only over the kept blocks (§3 states that the sparse branch of
 * RoLA, VSA and SLA is exact softmax on a retained block subset).  The paper
 * leaves the selector open (a top-k rule or block-level scores among other
 * choices); this library implements top-k over mean-pooled block scores.
 *
 * Conventions shared by every call
 *  - All tensor pointers are DEVICE pointers; descriptors, strides and sizes
 *    are host values.  The caller owns every buffer.  The library allocates
 *    no memory and keeps no pointer after a call returns.
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*; NULL
 *    is the default stream).  Inputs must stay alive until the stream has run.
 *  - Return value: SA_OK (0) or a negative sa_status.  Every argument check
 *    runs on the host before any HIP call, so an invalid call launches
 *    nothing and leaves all outputs untouched.  SA_ERR_LAUNCH reports a HIP
 *    launch error (hipGetLastError after the launches).
 *  - bf16 tensors are indexed [batch][head][token][channel] through the
 *    element strides in the descriptor; channels are contiguous; every stride
 *    must be a multiple of 8 elements and every pointer 16-byte aligned.
 *  - Inputs with NaN or Inf are outside the contract (results undefined).
 *  - Calls are reentrant; overlapping calls that share a workspace race.
 */
#ifndef SPARSE_ATTN_H
#define SPARSE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPARSE_ATTN_VERSION 100 /* 1.0.0 */

typedef enum {
  SA_OK = 0,
  SA_ERR_INVALID_ARG = -1, /* null pointer, bad size, misaligned pointer or stride */
  SA_ERR_UNSUPPORTED = -2, /* head_dim != 128, block not in {64, 128}, ... */
  SA_ERR_WORKSPACE = -3,   /* ws_bytes smaller than sparse_attn_workspace_size() */
  SA_ERR_LAUNCH = -4,      /* a HIP launch failed */
  SA_ERR_DEVICE = -5       /* no usable gfx950 device */
} sa_status;

/* Selection modes of sparse_attn_select. */
enum {
  SA_SELECT_ROW_TOPK = 0, /* every query block keeps exactly `budget` key blocks */
  SA_SELECT_HEAD_TOPK = 1 /* ragged: `budget` (query, key) block pairs per head */
};

/* Workspace consumers (second argument of sparse_attn_workspace_size):
 * SA_OP_SELECT is the row mode of sparse_attn_select, SA_OP_SELECT_HEAD its
 * whole-head mode. */
enum {
  SA_OP_SELECT = 0,
  SA_OP_SCHEDULE = 1,
  SA_OP_COMP_STATE = 2,
  SA_OP_BWD = 3,
  SA_OP_SELECT_HEAD = 4
};

/*
 * Problem descriptor (host struct).
 *  seqlen      tokens L of the flattened spatiotemporal sequence (>= 1)
 *  head_dim    d; must be 128
 *  block       tokens per query block and per key block: 64 (the paper's
 *              64x64 blocks, appendix "Training Details") or 128
 *  *_stride    element strides of (batch, head, token) for q, k, v, o
 *  softmax_scale  tau in softmax(tau * q.k); 0 selects fp32(1/sqrt(head_dim))
 * Blocks: nqb = nkb = ceil(seqlen / block); the last block holds the
 * remainder tokens and is a regular candidate.
 */
typedef struct {
  int32_t batch, heads, seqlen, head_dim, block;
  int64_t q_stride[3];
  int64_t k_stride[3];
  int64_t v_stride[3];
  int64_t o_stride[3];
  float softmax_scale;
  /* Causal window (paper §1: the sparse attention restricted to a causal
   * window for auto-regressive generation).  Tokens form chunks of
   * causal_chunk consecutive tokens (the latent frames generated together);
   * query t in chunk c = t / causal_chunk attends only keys of chunks
   * [c - causal_window + 1, c] (causal_window 0: every earlier chunk).
   * causal_chunk 0 (with causal_window 0) leaves attention unrestricted.
   * With a window, sparse_attn_select (row mode) ranks only the candidate
   * key blocks (those holding an allowed key of some query of the block) and
   * keeps min(budget, candidates) of them (cnt says how many; the rest of the
   * row is -1); the forward calls mask every score outside a query's allowed
   * keys, and a row left with none gets O = 0 and LSE = -inf; the backward
   * takes the same window; the compensation calls keep one state per chunk
   * (see sparse_attn_comp_state).  The whole-head selection mode returns
   * SA_ERR_UNSUPPORTED with a window.  Negative values, or a window without
   * chunks: SA_ERR_INVALID_ARG. */
  int32_t causal_chunk;
  int32_t causal_window;
} sparse_attn_desc;

/* SPARSE_ATTN_VERSION of the built library. */
int sparse_attn_version(void);

/* Static text for a status code. */
const char* sparse_attn_status_str(int status);

/* Key blocks kept per query block for a keep ratio in basis points
 * (1000 = 10%): ceil(keep_bp * nkb / 10000) clamped to [1, nkb]
 * (sparsity = 1 - k / nkb, paper §2 "Block sparsity").  Returns -1 when
 * keep_bp < 1 or nkb < 1. */
int32_t sparse_attn_keep_count(int32_t keep_bp, int32_t nkb);

/* Bytes of device workspace that `op` needs for this problem; `kmax` is the
 * row stride of the index list (ignored for SA_OP_SELECT and
 * SA_OP_SELECT_HEAD).  Returns 0 for an invalid descriptor or op.
 * Row-mode selection with nkb <= 1192 keeps the block scores on chip and
 * needs B*H*(2048*nkb + 16384*ceil(nkb/32) + 4*nkb) bytes; above that, and
 * in the whole-head mode, the fp64 score matrix (8*nkb^2 bytes per head) is
 * part of it. */
size_t sparse_attn_workspace_size(const sparse_attn_desc* desc, int32_t op, int32_t kmax);

/*
 * Block selection M_phi (paper §2 Eq. comp-sparse; §4.3 keeps mask
 * selection in BF16, so it reads the bf16 Q and K).
 *   score s_ij = (sum_{t in I_i} q_t) . (sum_{u in J_j} k_u) / (n_i n_j),
 * the mean unscaled logit of block (i, j), pooled and dotted in fp64.  The
 * row mode with nkb <= 1192 ranks bf16-matrix-core approximations of the
 * scores whose error is bounded, and rescores in fp64 the blocks whose bound
 * reaches across the k-th score, so its lists are those of the fp64 scores.
 *  q, k    bf16 [B][H][L][d] via desc strides (o_stride and v_stride unused)
 *  mode    SA_SELECT_ROW_TOPK: each query block keeps the `budget` key blocks
 *          with the largest score under (score desc, block index asc);
 *          1 <= budget <= nkb <= kmax is required.
 *          SA_SELECT_HEAD_TOPK: per (batch, head), `budget` block pairs in
 *          total (nqb <= budget <= nqb * nkb): every query block first keeps
 *          its best key block, then the remaining pairs go by (score desc,
 *          query block asc, key block asc).  A row that would keep more than
 *          kmax blocks (kmax >= 1, the list stride) keeps its kmax best by
 *          (score desc, key block asc); the pairs so dropped are not
 *          replaced, so cnt then sums to less than budget.
 *  idx     int32 [B][H][nqb][kmax] out: kept key-block indices, strictly
 *          ascending in the first cnt entries, -1 after them
 *  cnt     int32 [B][H][nqb] out: number of kept blocks per query block
 *  ws      device workspace of ws_bytes >= sparse_attn_workspace_size(SA_OP_SELECT)
 *          for SA_SELECT_ROW_TOPK, (SA_OP_SELECT_HEAD) for SA_SELECT_HEAD_TOPK
 */
int sparse_attn_select(const sparse_attn_desc* desc, const void* q, const void* k,
                       int32_t mode, int64_t budget, int32_t* idx, int32_t* cnt,
                       int32_t kmax, void* ws, size_t ws_bytes, void* stream);

/* Number of 64-row query tiles, B * H * ceil(L / 64): the length of the
 * launch order written by sparse_attn_schedule.  -1 for an invalid descriptor. */
int64_t sparse_attn_num_tiles(const sparse_attn_desc* desc);

/*
 * Work scheduling for the fused forward (ragged per-query-block work, the
 * selection lists of §2 Eq. comp-sparse being of unequal length in general).
 * Writes the launch order of the B*H*ceil(L/64) query tiles (tile t = (b*H +
 * h) * ceil(L/64) + row/64), a permutation of them.  The tiles are sorted by
 * cost class descending (longest first; stable, so equal classes keep raster
 * order), the class of a tile being 0 when its query block attends no key
 * tile and min(bit_length(key tiles), 15) otherwise, key tiles = 64-key tiles
 * = list length * block / 64.  Launch slot s then takes sorted position p(s),
 * which hands each XCD (slot mod 8) runs of 256 consecutive positions: in
 * groups of 2048 slots, p(s) = 2048 * (s / 2048) + 256 * (s mod 8) +
 * (s mod 2048) / 8, and the slots of a last partial group keep p(s) = s.
 * Only performance depends on the order: the forward's results are the same
 * bits with any order (or none).
 *  cnt     int32 [B][H][nqb] list lengths (clamped to [0, kmax])
 *  order   int32 [sparse_attn_num_tiles(desc)] out
 *  ws      ws_bytes >= sparse_attn_workspace_size(SA_OP_SCHEDULE)
 */
int sparse_attn_schedule(const sparse_attn_desc* desc, const int32_t* cnt, int32_t kmax,
                         int32_t* order, void* ws, size_t ws_bytes, void* stream);

/*
 * sparse_attn_schedule without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops that forbid
 * allocation): the same launch order as sparse_attn_schedule, bit for bit,
 * with its class counters in a 64 KiB device array inside the library, one
 * per GPU, held until the process ends.  The array of the current device is
 * used (the stream must belong to it); its address is looked up on the first
 * call on each device.  Every call on one GPU shares that array, so calls
 * that overlap on one GPU (other streams, other threads) race; calls
 * ordered on one stream do not.  No memory is allocated.
 *  cnt, kmax, order  as for sparse_attn_schedule
 * Errors: as sparse_attn_schedule, with SA_ERR_UNSUPPORTED when the problem
 * needs more than the array holds (more than 1,047,552 query tiles,
 * B * H * ceil(L / 64)), and SA_ERR_DEVICE when the array's device address
 * cannot be obtained. */
int sparse_attn_schedule_static(const sparse_attn_desc* desc, const int32_t* cnt, int32_t kmax,
                                int32_t* order, void* stream);

/*
 * Sparse branch O_s = A_M(Q, K, V) (paper §2 Eq. comp-sparse, §4.1), bf16.
 * For query block i with key-block list S_i = idx[b][h][i][0 .. cnt-1] and
 * U_i the tokens of those blocks, every query t of block i gets
 *   O_t = sum_{u in U_i} softmax_u(tau q_t.k_u) v_u,  LSE_t = log sum_u exp(tau q_t.k_u)
 * computed exactly (fp32 online softmax, bf16 MFMA products, fp32 accumulation).
 * List entries outside [0, nkb) are skipped and cnt is clamped to [0, kmax];
 * a query block with no valid entry gets O = 0 and LSE = -inf.
 *  q, k, v  bf16 via desc strides;  o  bf16 out via desc->o_stride
 *  idx/cnt  int32 [B][H][nqb][kmax] and [B][H][nqb], e.g. from
 *           sparse_attn_select; entries need not be ascending, but a block
 *           listed twice is attended twice (a caller error)
 *  order    launch order from sparse_attn_schedule for the same cnt, or NULL
 *           for plain raster order (results are identical either way)
 *  lse      fp32 [B][H][L] out, contiguous; may be NULL
 */
int sparse_attn_fwd(const sparse_attn_desc* desc, const void* q, const void* k,
                    const void* v, const int32_t* idx, const int32_t* cnt, int32_t kmax,
                    const int32_t* order, void* o, float* lse, void* stream);

/*
 * FP8 E4M3 (OCP e4m3fn) operand quantisation with one power-of-two scale per
 * block of desc->block tokens (the paper quantises its linear layers to E4M3,
 * §4.3; per-block scales for the attention operands are this library's choice).
 * For every (b, h, block): amax over the block's tokens and all channels,
 * scale = 2^e with the smallest integer e such that amax <= 448 * 2^e (scale 1
 * for an all-zero block), x8 = e4m3(x / scale) rounded to nearest even.
 *  x        bf16 [B][H][L][d] via x_stride (head_dim must be 128)
 *  x8       uint8 out, contiguous [B][H][L][d]
 *  scale    fp32 out, contiguous [B][H][nb]
 */
int sparse_attn_quant_fp8(const sparse_attn_desc* desc, const void* x, const int64_t x_stride[3],
                          uint8_t* x8, float* scale, void* stream);

/* Operands of sparse_attn_quant_fp8_tiles. */
enum { SA_FP8_K = 0, SA_FP8_V = 1 };

/*
 * The quantisation of sparse_attn_quant_fp8 (same codes, same scales), with
 * the codes written in the order in which the fp8 forward's matrix cores
 * consume K (operand SA_FP8_K) or V (SA_FP8_V), so that the forward reads
 * them with contiguous loads and no staging.  Per (b, h): T = ceil(L / 64)
 * tiles of 64 keys, 8192 bytes each; in tile t (keys 64 t .. 64 t + 63),
 * byte 16 c + e (c < 512, e < 16), with c = 64 f + l + 32 g (l < 32, g < 2):
 *   SA_FP8_K, f = 2 (2 rt + ks) + hf: key 64 t + 32 rt + l,
 *             channel 64 ks + 32 g + 16 hf + e
 *   SA_FP8_V, f = 2 dt + hf (dt < 4): channel 32 dt + l,
 *             key 64 t + 32 hf + 8 (e / 4) + 4 g + e % 4
 * Keys at or past L are code 0.
 *  x        bf16 [B][H][L][d] via x_stride (head_dim must be 128)
 *  operand  SA_FP8_K or SA_FP8_V (else SA_ERR_INVALID_ARG)
 *  x8       uint8 out, sparse_attn_fp8_tiles_bytes(desc) bytes, [B][H][T][8192]
 *  scale    fp32 out, contiguous [B][H][nb]
 */
int sparse_attn_quant_fp8_tiles(const sparse_attn_desc* desc, const void* x,
                                const int64_t x_stride[3], int32_t operand, uint8_t* x8,
                                float* scale, void* stream);

/* Bytes of one tile-layout operand, B * H * ceil(L / 64) * 8192; -1 for an
 * invalid descriptor. */
int64_t sparse_attn_fp8_tiles_bytes(const sparse_attn_desc* desc);

/*
 * Sparse branch on fp8 operands: the same result as sparse_attn_fwd computed
 * on the dequantised Q = sq * q8, K = sk * k8, V = sv * v8, with QK^T and PV on
 * the fp8 matrix cores; the probabilities are rounded to e4m3 for the PV
 * product.  q8 is contiguous [B][H][L][d] e4m3 as written by
 * sparse_attn_quant_fp8; k8 and v8 are in the tile layouts written by
 * sparse_attn_quant_fp8_tiles (SA_FP8_K, SA_FP8_V); sq, sk, sv are the
 * [B][H][nb] power-of-two scales of those calls.  o (via desc->o_stride),
 * lse, idx, cnt, kmax and order are as for sparse_attn_fwd.
 */
int sparse_attn_fwd_fp8(const sparse_attn_desc* desc, const uint8_t* q8, const float* sq,
                        const uint8_t* k8, const float* sk, const uint8_t* v8, const float* sv,
                        const int32_t* idx, const int32_t* cnt, int32_t kmax,
                        const int32_t* order, void* o, float* lse, void* stream);

/*
 * Compensation branch of compensated sparse attention (paper §2 Eq.
 * comp-sparse; §4.1 gives the low-rank branch with a token-wise gate):
 *   q~_i = R_r(p_i) silu(P_q q_i^norm),  k~_j = R_r(p_j) silu(P_k k_j^norm),
 *   C = sum_j k~_j v_j^T,  O_i = O_s,i + g_i * rms(O_s,i) * RMSNorm(q~_i^T C).
 * rank r must be 64 (the paper's compensation rank), else SA_ERR_UNSUPPORTED.
 * R_r rotates coordinate pairs (2m, 2m+1), m < r/2, as (a, b) -> (a c - b s,
 * a s + b c) with (c, s) = rope[token][m]; rope is fp32 [L][r/2][2], shared by
 * all heads (the caller's rotary schedule, e.g. the first r coordinates of the
 * backbone's 3D RoPE).  P_q, P_k are bf16 [H][r][d] row-major.  silu(x) =
 * x sigmoid(x); RMSNorm(y) = y / sqrt(mean_d y^2 + eps) * gamma; rms(x) =
 * sqrt(mean_d x^2).  Products run on bf16 operands with fp32 accumulation.
 * Under a causal window in the descriptor (causal_chunk > 0) the branch sees
 * the keys the sparse branch sees: query t in chunk c uses the state C_c
 * summed over the keys of chunks [c - causal_window + 1, c] (every chunk up
 * to c for causal_window 0), one state per chunk (paper §1, auto-regressive
 * extension).
 */

/* Low-rank state C for every (b, h) (and causal chunk), stored transposed.
 *  k_norm  bf16 [B][H][L][d] via kn_stride (the backbone's normalised keys)
 *  v       bf16 via desc->v_stride
 *  state   fp32 out, contiguous [B][H][nc][d][r]: state[b][h][k][c][m] =
 *          C_k[m][c], nc = ceil(L / causal_chunk) under a window, else 1
 *  ws      ws_bytes >= sparse_attn_workspace_size(SA_OP_COMP_STATE)
 * Deterministic: partial sums over fixed token chunks added in a fixed order. */
int sparse_attn_comp_state(const sparse_attn_desc* desc, int32_t rank, const void* k_norm,
                           const int64_t kn_stride[3], const void* v, const void* pk,
                           const float* rope, float* state, void* ws, size_t ws_bytes,
                           void* stream);

/* Gated output O = O_s + g * rms(O_s) * RMSNorm(q~^T C).
 *  q_norm  bf16 [B][H][L][d] via qn_stride
 *  state   fp32 [B][H][nc][d][r] from sparse_attn_comp_state (same descriptor
 *          window)
 *  gamma   fp32 [H][d] RMSNorm weight, or NULL for ones; eps >= 0
 *  gate    fp32 [B][H][L] via gate_stride (elements; 0 broadcasts)
 *  o_s     bf16 sparse-branch output via desc->o_stride
 *  o       bf16 out via desc->o_stride; may be o_s itself (in place) */
int sparse_attn_comp_out(const sparse_attn_desc* desc, int32_t rank, const void* q_norm,
                         const int64_t qn_stride[3], const void* pq, const float* rope,
                         const float* state, const float* gamma, float eps, const float* gate,
                         const int64_t gate_stride[3], const void* o_s, void* o, void* stream);

/*
 * Backward of the sparse branch (the gradients that the sparse model's
 * training needs, paper §2 and the Stage-1 warm-up of §4.4): for the lists
 * idx/cnt that the forward used, and its output o and log-sum-exp lse, with P = softmax(tau Q K_U^T)
 * over each query block's selected keys U:
 *   dV_U += P^T dO,  dS = P o (dO V_U^T - D),  D = rowsum(dO o O),
 *   dQ = tau dS K_U,  dK_U += tau dS^T Q.
 * Every key is covered: keys that no query block selected get dK = dV = 0,
 * query blocks with an empty list get dQ = 0.  With a causal window in the
 * descriptor (causal_chunk > 0) P is 0 outside each query's allowed keys, as
 * in the forward, and rows left without allowed keys (LSE = -inf) contribute
 * nothing.  Products are bf16 MFMA with fp32 accumulation; P and dS enter the
 * second products as bf16; outputs are bf16.  Deterministic (no
 * floating-point atomics).
 *  q, k, v, o, d_o   bf16 via desc strides (d_o laid out like o)
 *  lse               fp32 [B][H][L] natural log, as the forward wrote it
 *  idx, cnt, kmax    the forward's lists
 *  dq, dk, dv        bf16 out, laid out like q, k, v (desc strides)
 *  ws                ws_bytes >= sparse_attn_workspace_size(SA_OP_BWD)
 * Errors: SA_ERR_INVALID_ARG for null or misaligned pointers and bad
 * strides or lists; SA_ERR_UNSUPPORTED when a head of q, k, v or o spans
 * 4 GiB or more ((seqlen + 64) * token stride * 2 bytes, the kernels' 32-bit
 * row offsets); SA_ERR_WORKSPACE. */
int sparse_attn_bwd(const sparse_attn_desc* desc, const void* q, const void* k, const void* v,
                    const void* o, const void* d_o, const float* lse, const int32_t* idx,
                    const int32_t* cnt, int32_t kmax, void* dq, void* dk, void* dv, void* ws,
                    size_t ws_bytes, void* stream);

/*
 * W8A8 FP8 linear layers (paper §4.3: the attention and feed-forward
 * projections run on OCP e4m3 weights and activations; each weight output
 * channel has a static scale fixed offline, each activation token a scale
 * taken at run time, and the per-token quantisation is one fused pass).
 *
 * sparse_attn_quant_rows_fp8: per-row quantisation of bf16 x [rows][cols]
 * (row stride ldx elements) in one pass: a = max(max_k |x[r][k]|, 2^-100),
 * scale[r] = fp32(a / 448), q[r][k] = e4m3(fp32(x[r][k] * fp32(448 / a))),
 * rounded to nearest with ties to even (every fp32 step correctly rounded).
 * Used per token on activations and, once offline, per output channel on
 * weights [N][K].
 *  x      bf16 device pointer, 16-byte aligned; ldx >= cols, ldx % 8 == 0
 *  rows   >= 0 (0 launches nothing); cols >= 8, cols % 8 == 0
 *  q      uint8 [rows][cols] contiguous, 16-byte aligned (written)
 *  scale  fp32 [rows] (written)
 * Errors: SA_ERR_INVALID_ARG for null pointers, misalignment or bad sizes. */
int sparse_attn_quant_rows_fp8(const void* x, int64_t rows, int64_t cols, int64_t ldx, uint8_t* q,
                               float* scale, void* stream);

/*
 * sparse_attn_linear_w8a8: y[m][n] = bf16((sum_k dec(xq[m][k]) dec(wq[n][k]))
 * * sx[m] * sw[n] + bias[n]) with fp32 accumulation on the fp8 matrix cores
 * (the fp32 epilogue is fmaf(acc * sx[m], sw[n], bias[n]), rounded to nearest
 * even bf16).
 *  xq, sx   activation codes [M][K] (row stride ldx bytes) and scales [M], as
 *           written by sparse_attn_quant_rows_fp8
 *  wq, sw   weight codes [N][K] (row stride ldw bytes) and scales [N]
 *  bias     fp32 [N] or NULL
 *  y        bf16 [M][N], row stride ldy elements (written)
 * Layout rules: K % 128 == 0 and K >= 256; N % 8 == 0; M, N >= 0 (either 0
 * launches nothing); ldx, ldw >= K and multiples of 16; ldy >= N and a multiple
 * of 8; xq, wq, sw, bias and y 16-byte aligned; M, N < 2^31 and 256 * ldx,
 * 256 * ldw < 2^32.
 * Errors: SA_ERR_INVALID_ARG for null pointers, misalignment or bad sizes;
 * SA_ERR_UNSUPPORTED for sizes beyond the limits above. */
int sparse_attn_linear_w8a8(const uint8_t* xq, const float* sx, int64_t ldx, const uint8_t* wq,
                            const float* sw, int64_t ldw, const float* bias, void* y, int64_t ldy,
                            int64_t M, int64_t N, int64_t K, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SPARSE_ATTN_H */

// Host-side launchers of the gfx950 kernels (internal to the library; the
// public C ABI lives in include/sparse_attn.h).  Arguments have been checked
// by the caller; every launcher only enqueues work on `stream`.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sa {

struct Strides {
  int64_t b, h, n;  // elements per batch, head, token
};

struct Shape {
  int B, H, N, block, nb;  // nb = ceil(N / block) query blocks = key blocks
  // causal window: query t (chunk t / causal_chunk) sees the keys of chunks
  // [c - causal_window + 1, c] (causal_window 0: every earlier chunk);
  // causal_chunk 0: no restriction
  int causal_chunk = 0, causal_window = 0;
};

// Allowed key tokens [lo, hi) of query token t under the causal window.
__host__ __device__ inline int causal_lo(const Shape& s, int t) {
  if (s.causal_chunk <= 0 || s.causal_window == 0) return 0;
  const int c = t / s.causal_chunk - s.causal_window + 1;
  return c > 0 ? c * s.causal_chunk : 0;
}
__host__ __device__ inline int causal_hi(const Shape& s, int t) {
  if (s.causal_chunk <= 0) return s.N;
  const long long h = (long long)(t / s.causal_chunk + 1) * s.causal_chunk;
  return h < s.N ? (int)h : s.N;
}

// ---- selection -----------------------------------------------------------
// Workspace: qhat [B*H*nb*128] f64 | khat [same] | then, row mode with
// nb <= 1192, the split operands and norms of the fused kernel, otherwise the
// scores [B*H*nb*nb] f64 (whole-head mode: and the radix-select state).
size_t select_workspace_bytes(const Shape& s);       // row mode
size_t select_head_workspace_bytes(const Shape& s);  // whole-head mode
hipError_t launch_select_row(const Shape& s, const void* q, Strides qs, const void* k,
                             Strides ks, int topk, int kmax, int32_t* idx, int32_t* cnt,
                             void* ws, hipStream_t stream);
hipError_t launch_select_head(const Shape& s, const void* q, Strides qs, const void* k,
                              Strides ks, int64_t budget, int kmax, int32_t* idx,
                              int32_t* cnt, void* ws, hipStream_t stream);

// ---- scheduling ----------------------------------------------------------
size_t schedule_workspace_bytes(const Shape& s);
int64_t num_query_tiles(const Shape& s);
// Writes the launch order of the 64-row query tiles (int32 [B*H*ceil(N/64)]).
hipError_t launch_schedule(const Shape& s, const int32_t* cnt, int kmax, int32_t* order,
                           void* ws, hipStream_t stream);
// Size of the file-scope device array that replaces the schedule workspace in
// the allocation-free entry point (one per GPU, held until the process ends).
constexpr size_t kStaticScheduleScratchBytes = 64 * 1024;
// Device address of the current GPU's copy of that array (looked up once per
// device); hipSuccess or the HIP error of the lookup.
hipError_t static_schedule_scratch(int32_t** out);

// ---- forward -------------------------------------------------------------
struct FwdArgs {
  const void* q;
  const void* k;
  const void* v;
  void* o;
  float* lse;
  Strides qs, ks, vs, os;
  const int32_t* idx;
  const int32_t* cnt;
  const int32_t* order;  // launch order of query tiles (may be null: natural)
  const float* sq;       // fp8 block scales (fp8 path only)
  const float* sk;
  const float* sv;
  int kmax;
  float softmax_scale;
};
hipError_t launch_fwd_bf16(const Shape& s, const FwdArgs& a, hipStream_t stream);
hipError_t launch_fwd_fp8(const Shape& s, const FwdArgs& a, hipStream_t stream);

// ---- compensation branch -------------------------------------------------
struct CompStateIn {
  const void* k_norm;  // bf16 [B][H][N][128] via kns
  const void* v;       // bf16 via vs
  const void* pk;      // bf16 [H][64][128]
  const float* rope;   // fp32 [N][32][2] (cos, sin)
  Strides kns, vs;
};
struct CompOutIn {
  const void* q_norm;  // bf16 via qns
  const void* pq;      // bf16 [H][64][128]
  const float* rope;
  const float* state;  // fp32 [B][H][chunks][128][64] (C^T, d-major)
  const float* gamma;  // fp32 [H][128] or null
  const float* gate;   // fp32 via gs
  const void* o_s;     // bf16 via oss
  void* o;             // bf16 via oss (may equal o_s)
  Strides qns, gs, oss;
  float eps;
};
// states per head: one per causal chunk, or 1 without a window
int comp_state_chunks(const Shape& s);
size_t comp_state_workspace_bytes(const Shape& s);
hipError_t launch_comp_state(const Shape& s, const CompStateIn& in, float* state, void* ws,
                             hipStream_t stream);
hipError_t launch_comp_out(const Shape& s, const CompOutIn& in, hipStream_t stream);

// ---- backward ------------------------------------------------------------
struct BwdIn {
  const void* q;
  const void* k;
  const void* v;
  const void* o;
  const void* dout;   // laid out like o
  const float* lse;   // [B][H][N] natural log, from the forward
  const int32_t* idx;
  const int32_t* cnt;
  void* dq;           // laid out like q
  void* dk;           // like k
  void* dv;           // like v
  Strides qs, ks, vs, os;
  int kmax;
  float softmax_scale;
};
// Workspace: D fp32 [B*H*N] (256-byte aligned) | bitmap u32 [B*H][nb][ceil(nb/32)]
size_t bwd_workspace_bytes(const Shape& s);
hipError_t launch_bwd(const Shape& s, const BwdIn& in, void* ws, hipStream_t stream);

// ---- fp8 quantisation ----------------------------------------------------
hipError_t launch_quant_fp8(const Shape& s, const void* x, Strides xs, uint8_t* x8,
                            float* scale, hipStream_t stream);
// The same codes in the fp8 forward's K (is_v false) or V operand order:
// [B*H][ceil(N / 64)][8192 bytes].
hipError_t launch_quant_fp8_tiles(const Shape& s, const void* x, Strides xs, bool is_v,
                                  uint8_t* x8, float* scale, hipStream_t stream);

// ---- W8A8 fp8 linear layers -----------------------------------------------
// Per-row e4m3 quantisation of bf16 x [rows][cols] (row stride ldx elements)
// into q [rows][cols] (contiguous) and fp32 scale [rows].
hipError_t launch_quant_rows_fp8(const void* x, int64_t ldx, int64_t rows, int cols, uint8_t* q,
                                 float* scale, hipStream_t stream);
struct LinearIn {
  const uint8_t* xq;  // [M][K] activation codes, row stride ldx bytes
  const float* sx;    // [M]
  const uint8_t* wq;  // [N][K] weight codes, row stride ldw bytes
  const float* sw;    // [N]
  const float* bias;  // [N] or null
  void* y;            // bf16 [M][N], row stride ldy elements
  int64_t ldx, ldw, ldy;
  int64_t M, N, K;
  int group_m;        // tile rows per launch-order group (0: default)
};
hipError_t launch_linear_w8a8(const LinearIn& in, hipStream_t stream);

}  // namespace sa

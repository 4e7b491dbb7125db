// Compensation branch and gate epilogue of compensated sparse attention on
// gfx950 (paper §2 Eq. comp-sparse; §4.1 defines the branch):
//
//   q~_i = R_r(p_i) silu(P_q q_i^norm),   k~_j = R_r(p_j) silu(P_k k_j^norm)
//   C = sum_j k~_j v_j^T                       (rank r = 64, per (batch, head))
//   O_i = O_s,i + g_i * rms(O_s,i) * RMSNorm(q~_i^T C)
//
// R_r rotates consecutive coordinate pairs (2m, 2m+1) by angles given as a
// (cos, sin) table per token and pair.  Three launches:
//   comp_state  : per (head, chunk of 2048 tokens) the projection k_norm P_k^T
//                 on the matrix cores in the layout that keeps tokens inside a
//                 lane (so k~ is directly the B operand of the next product),
//                 silu and the rotation (the partner coordinate of a pair sits
//                 in the neighbouring lane: one DPP swap), then
//                 C^T += V^T K~ with V^T read transposed from LDS; the four
//                 waves' partials are summed through LDS in a fixed order.
//   comp_reduce : the chunk partials of a head summed in chunk order -> C^T
//                 (fp32, d-major: row d holds the r values of C[.][d]).
//   comp_out    : per (head, 1024 tokens, in tiles of 128) the projection P_q q_norm^T in the
//                 layout that keeps one token per lane, silu and rotation,
//                 O_lr^T = C^T q~^T against a bf16 hi + lo copy of C^T in LDS, then
//                 RMSNorm, the gate and the sum with O_s, all per lane.
// The projections multiply the bf16 inputs exactly (fp32 accumulation).  In
// the two low-rank products the fp32 operands k~, q~ and C are each split as
// hi + lo with hi = bf16(x) and lo = bf16(x - hi) (about 16 significant
// bits), and the products taken as hi.hi + hi.lo + lo.hi on the bf16 matrix
// cores, so the state and O_lr carry close to fp32 accuracy; silu, rotation
// and the normalisations are fp32.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kRank = 64;
constexpr int kSub = 128;               // tokens per sub-tile (4 waves x 32)
constexpr int kChunk = 1024;            // tokens per state workgroup
constexpr int kReduceSplit = 32;        // workgroups per head in the chunk reduction
static_assert(kReduceSplit * 256 == 64 * 128, "one reduction thread per state element");
constexpr int kStateElems = kRank * kHeadDim;
constexpr int kRopeBytes = kRank / 2 * 2 * 4;  // (cos, sin) fp32 per pair, per token
constexpr int kVRow = kHeadDim * 2;     // bf16 V row in LDS
constexpr int kCtStride = 72;           // bf16 per C^T row in LDS (64 + 8 padding)

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }
// silu(x) = x sigmoid(x), the reciprocal by v_rcp_f32 (1 ulp) rather than
// a full-precision division
__device__ __forceinline__ float silu(float x) {
  return x * __builtin_amdgcn_rcpf(1.f + __expf(-x));
}

// Exchange words 0, 1 of lanes 32..63 with words 2, 3 of lanes 0..31
// (v_permlane32_swap).  With lane l (< 32) holding channels c..c+7 of a row
// and lane l + 32 channels c+8..c+15, afterwards lane l holds c..c+3 and
// c+8..c+11, lane l + 32 holds c+4..c+7 and c+12..c+15; applied again it
// restores the contiguous halves.
__device__ __forceinline__ u32x4 swap_quads(u32x4 w) {
  const auto s0 = __builtin_amdgcn_permlane32_swap(w[0], w[2], false, false);
  const auto s1 = __builtin_amdgcn_permlane32_swap(w[1], w[3], false, false);
  const u32x4 r = {s0[0], s1[0], s0[1], s1[1]};
  return r;
}

// Lane id read afresh: LDS addresses derived from it inside a loop are not
// loop invariants, so the compiler cannot hoist every read of data that
// stays in LDS out of the loop (and hold it all in registers).
__device__ __forceinline__ int fresh_lane() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// 16-byte-chunk swizzle of the V rows in LDS (as in the forward): conflict-free
// for the transpose reads of 4 rows x 4 chunks per half-wave.
__device__ __forceinline__ int swz_v(int row, int chunk) { return chunk ^ ((row & 3) << 2); }

struct StateArgs {
  const uint16_t* kn;
  const uint16_t* v;
  const uint16_t* pk;
  const float* rope;
  float* partial;  // [BH][chunks][kStateElems], lane-register order
  Strides kns, vs;
  int H, N, chunks;
};

// partial element e = ((dt*2 + nb)*16 + reg)*64 + lane holds C^T[d][r] with
// r = 32 nb + (lane & 31), d = 32 dt + 8 (reg >> 2) + 4 (lane >> 5) + (reg & 3).
__global__ __launch_bounds__(256) void comp_state_kernel(StateArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t vt[kSub * kVRow];
  const int bh = blockIdx.x, chunk = blockIdx.y;  // heads vary fastest: rope rows shared in L2
  const int b = bh / a.H, h = bh - b * a.H;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int g = lane >> 5, l32 = lane & 31;
  const int t_begin = chunk * kChunk, t_end = min(t_begin + kChunk, a.N);

  const uint32_t kst = (uint32_t)a.kns.n * 2, vst = (uint32_t)a.vs.n * 2;
  const auto kr = make_rsrc(a.kn + b * a.kns.b + h * a.kns.h, (uint32_t)(a.N - 1) * kst + 256u);
  const auto vr = make_rsrc(a.v + b * a.vs.b + h * a.vs.h, (uint32_t)(a.N - 1) * vst + 256u);
  const auto rr = make_rsrc(a.rope, (uint32_t)a.N * kRopeBytes);

  // P_k as B operand of k_norm P_k^T: column r = l32 + 32 nb, k = d 16 ks + 8 g .. +7
  bf16x8 pkf[2][8];
  const uint16_t* pkh = a.pk + (int64_t)h * kStateElems;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      pkf[nb][ks] = as_bf16x8(ld16(pkh + (l32 + 32 * nb) * kHeadDim + 16 * ks + 8 * g));

  f32x16 acc[4][2];  // C^T: [dt][nb]
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[dt][nb][r] = 0.f;

  // transpose-read addresses of V^T (rows = this wave's tokens, as the
  // forward's keys): lane 16G + 4e + q reads the 8-byte chunk of token
  // 32 wave + 16 s + 8 hf + 4 (G>>1) + e at channels 32 dt + 16 (G&1) + 4 q
  const int G = lane >> 4, e4 = (lane >> 2) & 3, q4 = lane & 3;
  const int vrow0 = 32 * wave + 4 * (G >> 1) + e4;

  // k_norm as A operand (token tw + l32, channels 16 ks + 8 g .. +7) and the
  // sub-tile's V rows (thread t moves chunks e = t + 256 m -> row e/16, chunk
  // e%16); the next sub-tile's are fetched while the current one is computed
  bf16x8 kf[8];
  u32x4 vrow[8];
  auto load_kv = [&](int t0) {
    const int tw = t0 + 32 * wave;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      kf[ks] = as_bf16x8(buf_ld16(kr, (uint32_t)(tw + l32) * kst + (16 * ks + 8 * g) * 2));
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int e = t + 256 * m, row = e >> 4, ch = e & 15;
      vrow[m] = buf_ld16(vr, (uint32_t)(t0 + row) * vst + ch * 16);
    }
  };
  if (t_begin < t_end) load_kv(t_begin);

  for (int t0 = t_begin; t0 < t_end; t0 += kSub) {
    const int tw = t0 + 32 * wave;
    // (cos, sin) of this lane's pair m = (32 nb + l32) / 2 at its 16 tokens
    // tw + 8 j + 4 g + rr
    float2 cs[2][16];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int tok = tw + 8 * (i >> 2) + 4 * g + (i & 3);
        const uint32_t off = (uint32_t)tok * kRopeBytes + (uint32_t)((32 * nb + l32) >> 1) * 8u;
        const u32x2 w = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rr, off, 0, 0));
        cs[nb][i] = make_float2(__uint_as_float(w[0]), __uint_as_float(w[1]));
      }
    __syncthreads();  // every wave is done reading the previous sub-tile's V
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int e = t + 256 * m, row = e >> 4, ch = e & 15;
      *reinterpret_cast<u32x4*>(vt + row * kVRow + swz_v(row, ch) * 16) = vrow[m];
    }

    // projection k_norm P_k^T: lane holds column r = 32 nb + l32 of tokens
    // 8 j + 4 g + rr (register 4 j + rr)
    f32x16 pr[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) pr[nb][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks)
        pr[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks], pkf[nb][ks], pr[nb], 0, 0, 0);
    }
    if (t0 + kSub < t_end) load_kv(t0 + kSub);  // prefetch the next sub-tile
    // silu, then the rotation of pair (r & ~1, r | 1): the partner column is
    // the neighbouring lane (DPP quad_perm 1,0,3,2)
    const bool odd = (l32 & 1) != 0;
    // K~ as B operand, split hi + lo: [nb][k-step s], tokens 16 s + 4 g + rr, 16 s + 8 + 4 g + rr
    bf16x8 kt[2][2], kl[2][2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      float y[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float x = silu(pr[nb][i]);
        const float o = __int_as_float(
            __builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
        const float c = cs[nb][i].x, s = cs[nb][i].y;
        // even r: (x, o) = (a, b) -> a c - b s;  odd r: (o, x) = (a, b) -> a s + b c
        y[i] = odd ? fmaf(o, s, x * c) : fmaf(x, c, -o * s);
      }
#pragma unroll
      for (int sk = 0; sk < 2; ++sk)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const __bf16 hi = (__bf16)y[8 * sk + e];
          kt[nb][sk][e] = hi;
          kl[nb][sk][e] = (__bf16)(y[8 * sk + e] - (float)hi);
        }
    }
    __syncthreads();  // the sub-tile's V rows are in LDS

    // C^T += V^T K~ over this wave's 32 tokens
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int lc = 4 * dt + 2 * (G & 1) + (q4 >> 1);
      const int half = (q4 & 1) * 8;
#pragma unroll
      for (int sk = 0; sk < 2; ++sk) {
        u32x4 vv;
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int row = vrow0 + 16 * sk + 8 * hf;
          const i16x4 tr = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) i16x4*)(vt + row * kVRow + swz_v(row, lc) * 16 +
                                                         half));
          const u32x2 tw2 = __builtin_bit_cast(u32x2, tr);
          vv[2 * hf] = tw2[0];
          vv[2 * hf + 1] = tw2[1];
        }
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          acc[dt][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), kt[nb][sk],
                                                                acc[dt][nb], 0, 0, 0);
          acc[dt][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), kl[nb][sk],
                                                                acc[dt][nb], 0, 0, 0);
        }
      }
    }
  }

  // sum the four waves' partials in wave order through LDS, then store
  float* red = reinterpret_cast<float*>(vt);  // 32 KB = kStateElems floats
  for (int w = 0; w < 4; ++w) {
    __syncthreads();
    if (wave == w) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int e = ((dt * 2 + nb) * 16 + r) * 64 + lane;
            red[e] = w == 0 ? acc[dt][nb][r] : red[e] + acc[dt][nb][r];
          }
    }
  }
  __syncthreads();
  float* out = a.partial + ((int64_t)bh * a.chunks + chunk) * kStateElems;
  for (int e = t; e < kStateElems; e += 256) out[e] = red[e];
}

// C^T[bh][d][r] = sum over chunks (in chunk order) of the partials; each
// workgroup sums 256 of a head's elements.
__global__ __launch_bounds__(256) void comp_reduce_kernel(const float* __restrict__ partial,
                                                          int chunks, float* __restrict__ state) {
  const int bh = blockIdx.x;
  const int e = blockIdx.y * 256 + threadIdx.x;
  const float* src = partial + (int64_t)bh * chunks * kStateElems + e;
  float s = 0.f;
  for (int c = 0; c < chunks; ++c) s += src[(int64_t)c * kStateElems];
  const int lane = e & 63, reg = (e >> 6) & 15, blk = e >> 10;  // blk = dt * 2 + nb
  const int dt = blk >> 1, nb = blk & 1;
  const int r = 32 * nb + (lane & 31);
  const int d = 32 * dt + 8 * (reg >> 2) + 4 * (lane >> 5) + (reg & 3);
  state[(int64_t)bh * kStateElems + d * kRank + r] = s;
}

struct OutArgs {
  const uint16_t* qn;
  const uint16_t* pq;
  const float* rope;
  const float* state;
  const float* gamma;  // [H][d] or null
  const float* gate;
  const uint16_t* os;
  uint16_t* o;
  Strides qns, gs, oss;
  int H, N;
  float eps;
};

// LDS position of rank index r in a C^T row: within each group of 16 the
// middle quads swap, so that lane group g reads the 8 indices
// {16s + 4g + 0..3, 16s + 8 + 4g + 0..3} of k-step s as one 16-byte chunk.
__device__ __forceinline__ int ct_pos(int r) {
  const int q = r & 15, quad = q >> 2;
  const int nq = quad == 1 ? 2 : (quad == 2 ? 1 : quad);
  return (r & ~15) + 4 * nq + (q & 3);
}

// Per-token inputs of one 128-token tile for this lane's token `tok`
// (clamped into the sequence): q_norm as the B operand of the projection
// (channels 16 ks + 8 g .. +7), O_s (after swap_quads: channels
// 32 dt + 8 j + 4 g + {0..3} in osw[dt][j]) and the gate.
__device__ __forceinline__ void load_tok(const OutArgs& a, int b, int h, int tokc, int g,
                                         bf16x8 (&qf)[8], u32x2 (&osw)[4][4], float& gv) {
  const uint16_t* qrow = a.qn + b * a.qns.b + h * a.qns.h + (int64_t)tokc * a.qns.n;
#pragma unroll
  for (int ks = 0; ks < 8; ++ks) qf[ks] = as_bf16x8(ld16(qrow + 16 * ks + 8 * g));
  // 16-byte loads of channels 32 dt + 16 jp + 8 g .. +7, regrouped across
  // the lane pair by swap_quads (done by the caller once the loads landed)
  const uint16_t* osrow = a.os + b * a.oss.b + h * a.oss.h + (int64_t)tokc * a.oss.n;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int jp = 0; jp < 2; ++jp) {
      const u32x4 w = ld16(osrow + 32 * dt + 16 * jp + 8 * g);
      osw[dt][2 * jp] = u32x2{w[0], w[1]};
      osw[dt][2 * jp + 1] = u32x2{w[2], w[3]};
    }
  gv = a.gate[b * a.gs.b + h * a.gs.h + (int64_t)tokc * a.gs.n];
}

// One workgroup per (head, kOutTiles tiles of 128 tokens): C^T (as bf16 hi +
// lo) and P_q are staged into LDS once, then the tiles stream through, the
// next tile's per-token loads issued before the current tile is computed.
constexpr int kOutTiles = 8;

__global__ __launch_bounds__(256, 2) void comp_out_kernel(OutArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ct[kHeadDim * kCtStride];   // C^T hi
  __shared__ __attribute__((aligned(16))) uint16_t ctl[kHeadDim * kCtStride];  // C^T lo
  // P_q rows (r, 256 bytes each); 16-byte chunk c of row r at slot c ^ (r & 15)
  __shared__ __attribute__((aligned(16))) uint8_t pqs[kRank * kHeadDim * 2];
  __shared__ __attribute__((aligned(16))) float gam_s[kHeadDim];  // RMSNorm weight (1 if none)
  const int bh = blockIdx.x;
  const int b = bh / a.H, h = bh - b * a.H;
  const int ntiles = (a.N + kSub - 1) / kSub;
  const int tile0 = blockIdx.y * kOutTiles, tile_end = min(tile0 + kOutTiles, ntiles);
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int g = lane >> 5, l32 = lane & 31;

  // the first tile's per-token loads are issued first, so their latency
  // overlaps the staging of C^T and P_q
  bf16x8 qf[8];
  u32x2 osw[4][4];
  float gv;
  load_tok(a, b, h, min(tile0 * kSub + 32 * wave + l32, a.N - 1), g, qf, osw, gv);

  // C^T of this head as bf16 hi + lo into LDS: thread t converts quads of
  // 4 consecutive r (16-byte loads) and stores each as 8 bytes at its
  // permuted position
  const float* st = a.state + (int64_t)bh * kStateElems;
#pragma unroll
  for (int m = 0; m < kStateElems / 4 / 256; ++m) {
    const int qd = t + 256 * m;              // quad index: d = qd / 16, r = 4 (qd % 16)
    const int d = qd >> 4, r = (qd & 15) * 4;
    const f32x4 x = *reinterpret_cast<const f32x4*>(st + 4 * qd);
    u32x2 hw, lw;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const __bf16 h0 = (__bf16)x[2 * u], h1 = (__bf16)x[2 * u + 1];
      const __bf16 l0 = (__bf16)(x[2 * u] - (float)h0), l1 = (__bf16)(x[2 * u + 1] - (float)h1);
      hw[u] = (uint32_t)__builtin_bit_cast(uint16_t, h0) |
              ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
      lw[u] = (uint32_t)__builtin_bit_cast(uint16_t, l0) |
              ((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16);
    }
    *reinterpret_cast<u32x2*>(ct + d * kCtStride + ct_pos(r)) = hw;
    *reinterpret_cast<u32x2*>(ctl + d * kCtStride + ct_pos(r)) = lw;
  }
  // P_q of this head: thread t moves 16-byte chunks e = t + 256 m
  const uint16_t* pqh = a.pq + (int64_t)h * kStateElems;
#pragma unroll
  for (int m = 0; m < kRank * 16 / 256; ++m) {
    const int e = t + 256 * m, r = e >> 4, c = e & 15;
    *reinterpret_cast<u32x4*>(pqs + r * 256 + ((c ^ (r & 15)) << 4)) = ld16(pqh + 8 * e);
  }
  if (t < kHeadDim) gam_s[t] = a.gamma ? a.gamma[(int64_t)h * kHeadDim + t] : 1.f;
  __syncthreads();  // C^T, P_q and the RMSNorm weight are in LDS

  for (int tile = tile0; tile < tile_end; ++tile) {
    const int tok = tile * kSub + 32 * wave + l32;  // this lane's token
    // (cos, sin) of this lane's pairs: pairs (rr = 0, 1) and (2, 3) of each
    // (rb, j) are pairs m = 16 rb + 4 j + 2 g + {0, 1}, 16 contiguous bytes.
    // Issued before the next tile's loads, so waiting for them does not wait
    // for those.
    const float* rope_t = a.rope + (int64_t)min(tok, a.N - 1) * (kRank / 2) * 2;
    f32x4 csn[2][4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        csn[rb][j] = *reinterpret_cast<const f32x4*>(rope_t + 2 * (16 * rb + 4 * j + 2 * g));
    // the next tile's per-token inputs (on the last tile the current one's
    // again, L2-resident: the loads are issued on every path, so the waits
    // the compiler places for the loads above count them)
    bf16x8 qn[8];
    u32x2 on[4][4];
    float gn;
    load_tok(a, b, h, min(tile + 1 < tile_end ? tok + kSub : tok, a.N - 1), g, qn, on, gn);

    // projection P_q q_norm^T: lane holds token `tok`, rank indices
    // 32 rb + 8 j + 4 g + rr (P_q rows r = l32 + 32 rb as the A operand)
    const int ln = fresh_lane(), fl32 = ln & 31, fg = ln >> 5;
    f32x16 pr[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) pr[rb][r] = 0.f;
      const int prow = fl32 + 32 * rb;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const bf16x8 pf = as_bf16x8(*reinterpret_cast<const u32x4*>(
            pqs + prow * 256 + (((2 * ks + fg) ^ (prow & 15)) << 4)));
        pr[rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf, qf[ks], pr[rb], 0, 0, 0);
      }
    }
    // silu and rotation; q~^T as B operand split hi + lo, k-step s: indices 16 s + 4 g + rr, 16 s + 8 + 4 g + rr
    bf16x8 qt[4], ql[4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 cj = csn[rb][j];
        float y[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) y[u] = silu(pr[rb][4 * j + u]);
        const float r0 = fmaf(y[0], cj[0], -y[1] * cj[1]);
        const float r1 = fmaf(y[0], cj[1], y[1] * cj[0]);
        const float r2 = fmaf(y[2], cj[2], -y[3] * cj[3]);
        const float r3 = fmaf(y[2], cj[3], y[3] * cj[2]);
        const int s2 = 2 * rb + (j >> 1), half = 4 * (j & 1);
        const float rv[4] = {r0, r1, r2, r3};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const __bf16 hi = (__bf16)rv[u];
          qt[s2][half + u] = hi;
          ql[s2][half + u] = (__bf16)(rv[u] - (float)hi);
        }
      }

    // O_lr^T = C^T q~^T: lane holds token `tok`, channels 32 dt + 8 j + 4 g + rr
    f32x16 y[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) y[dt][r] = 0.f;
      const uint16_t* crow = ct + (32 * dt + fl32) * kCtStride;
      const uint16_t* clrow = ctl + (32 * dt + fl32) * kCtStride;
#pragma unroll
      for (int s2 = 0; s2 < 4; ++s2) {
        const bf16x8 cf = as_bf16x8(*reinterpret_cast<const u32x4*>(crow + 16 * s2 + 8 * fg));
        const bf16x8 cl = as_bf16x8(*reinterpret_cast<const u32x4*>(clrow + 16 * s2 + 8 * fg));
        y[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cl, qt[s2], y[dt], 0, 0, 0);
        y[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cf, ql[s2], y[dt], 0, 0, 0);
        y[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cf, qt[s2], y[dt], 0, 0, 0);
      }
    }

    // RMSNorm of O_lr and rms of O_s over the 128 channels (64 here, 64 in lane l ^ 32)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int jp = 0; jp < 2; ++jp) {
        const u32x4 w = swap_quads(u32x4{osw[dt][2 * jp][0], osw[dt][2 * jp][1],
                                         osw[dt][2 * jp + 1][0], osw[dt][2 * jp + 1][1]});
        osw[dt][2 * jp] = u32x2{w[0], w[1]};
        osw[dt][2 * jp + 1] = u32x2{w[2], w[3]};
      }
    float ss_y = 0.f, ss_o = 0.f;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u32x2 w = osw[dt][j];
        const float o4[4] = {bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          ss_y = fmaf(y[dt][4 * j + u], y[dt][4 * j + u], ss_y);
          ss_o = fmaf(o4[u], o4[u], ss_o);
        }
      }
    ss_y += __shfl_xor(ss_y, 32, kWave);
    ss_o += __shfl_xor(ss_o, 32, kWave);
    const float rstd = 1.f / sqrtf(ss_y * (1.f / kHeadDim) + a.eps);
    const float rms_o = sqrtf(ss_o * (1.f / kHeadDim));
    const float coef = gv * rms_o * rstd;
    if (tok < a.N) {
      uint16_t* orow = a.o + b * a.oss.b + h * a.oss.h + (int64_t)tok * a.oss.n;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int jp = 0; jp < 2; ++jp) {
          u32x4 wo;
#pragma unroll
          for (int jj = 0; jj < 2; ++jj) {
            const int j = 2 * jp + jj;
            const int d0 = 32 * dt + 8 * j + 4 * g;
            const f32x4 gm = *reinterpret_cast<const f32x4*>(gam_s + d0);
            const u32x2 w = osw[dt][j];
            const float o4[4] = {bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
            float x[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) x[u] = fmaf(coef * y[dt][4 * j + u], gm[u], o4[u]);
            wo[2 * jj] = pack_bf16x2(x[0], x[1]);
            wo[2 * jj + 1] = pack_bf16x2(x[2], x[3]);
          }
          // back to 8 contiguous channels per lane: 32 dt + 16 jp + 8 g ..
          st16(orow + 32 * dt + 16 * jp + 8 * g, swap_quads(wo));
        }
    }
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) qf[ks] = qn[ks];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) osw[dt][j] = on[dt][j];
    gv = gn;
  }
}

}  // namespace

size_t comp_state_workspace_bytes(const Shape& s) {
  const int64_t chunks = (s.N + kChunk - 1) / kChunk;
  return (size_t)s.B * s.H * chunks * kStateElems * sizeof(float);
}

hipError_t launch_comp_state(const Shape& s, const CompStateIn& in, float* state, void* ws,
                             hipStream_t stream) {
  StateArgs a;
  a.kn = static_cast<const uint16_t*>(in.k_norm);
  a.v = static_cast<const uint16_t*>(in.v);
  a.pk = static_cast<const uint16_t*>(in.pk);
  a.rope = in.rope;
  a.partial = static_cast<float*>(ws);
  a.kns = in.kns;
  a.vs = in.vs;
  a.H = s.H;
  a.N = s.N;
  a.chunks = (s.N + kChunk - 1) / kChunk;
  comp_state_kernel<<<dim3(s.B * s.H, a.chunks), 256, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  comp_reduce_kernel<<<dim3(s.B * s.H, kReduceSplit), 256, 0, stream>>>(a.partial, a.chunks,
                                                                         state);
  return hipGetLastError();
}

hipError_t launch_comp_out(const Shape& s, const CompOutIn& in, hipStream_t stream) {
  OutArgs a;
  a.qn = static_cast<const uint16_t*>(in.q_norm);
  a.pq = static_cast<const uint16_t*>(in.pq);
  a.rope = in.rope;
  a.state = in.state;
  a.gamma = in.gamma;
  a.gate = in.gate;
  a.os = static_cast<const uint16_t*>(in.o_s);
  a.o = static_cast<uint16_t*>(in.o);
  a.qns = in.qns;
  a.gs = in.gs;
  a.oss = in.oss;
  a.H = s.H;
  a.N = s.N;
  a.eps = in.eps;
  const int ntiles = (s.N + kSub - 1) / kSub;
  comp_out_kernel<<<dim3(s.B * s.H, (ntiles + kOutTiles - 1) / kOutTiles), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace sa

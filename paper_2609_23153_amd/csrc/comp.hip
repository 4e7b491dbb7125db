// Compensation branch and gate epilogue of compensated sparse attention on
// gfx950 (paper §2 Eq. comp-sparse; §4.1 defines the branch):
//
//   q~_i = R_r(p_i) silu(P_q q_i^norm),   k~_j = R_r(p_j) silu(P_k k_j^norm)
//   C = sum_j k~_j v_j^T                       (rank r = 64, per (batch, head))
//   O_i = O_s,i + g_i * rms(O_s,i) * RMSNorm(q~_i^T C)
//
// R_r rotates consecutive coordinate pairs (2m, 2m+1) by angles given as a
// (cos, sin) table per token and pair.  Three launches:
//   comp_state  : per (head, chunk of 1024 tokens, in sub-tiles of 128) the
//                 projection P_k k_norm^T on the matrix cores in the layout
//                 that keeps one token per lane (both coordinates of a
//                 rotation pair in one lane), silu and the rotation, K~ to
//                 LDS, then C^T += V^T K~ with V^T and K~ read transposed
//                 from LDS, wave w owning rows 32 w .. of C^T.
//   comp_reduce : the chunk partials of a head summed in chunk order -> C^T
//                 (fp32, d-major: row d holds the r values of C[.][d]).
//   comp_out    : per (head, 1024 tokens, in tiles of 128) the projection
//                 P_q q_norm^T in the same one-token-per-lane layout, silu
//                 and rotation, O_lr^T = C^T q~^T against a bf16 hi + lo copy
//                 of C^T in LDS, then RMSNorm, the gate and the sum with O_s,
//                 all per lane.
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
// Two fp32 values as packed bf16, rounded to nearest even by the hardware
// conversion (v_cvt_pk_bf16_f32): one instruction per pair.
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  const bf16x2_t t = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, t);
}

// x0, x1 split as packed bf16 hi and lo pairs {hi, lo}: hi = bf16(x),
// lo = bf16(x - hi) (the hi values unpack to fp32 exactly by a shift and a
// mask).
__device__ __forceinline__ u32x2 split_pair(float x0, float x1) {
  const uint32_t hw = cvt_pk_bf16(x0, x1);
  return u32x2{hw, cvt_pk_bf16(x0 - bf16_lo(hw), x1 - bf16_hi(hw))};
}

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
  float* partial;  // [BH][nc * nsub][kStateElems], lane-register order
  Strides kns, vs;
  int H, N;
  int span;  // tokens per causal chunk (N without a window)
  int nc;    // causal chunks, ceil(N / span)
  int nsub;  // 1024-token sub-chunks per causal chunk, ceil(span / 1024)
};

// K~ sub-tile in LDS: [token][r] bf16, 128-byte rows; 16-byte chunk c of
// row t at slot c ^ kt_swz(t): conflict-free for the transposed reads
// (4 rows x 4 chunks per half-wave: rows t, t + 2 land in opposite halves of
// the row) and 2-way for the row writes (32 rows, one chunk each).
__device__ __forceinline__ int kt_swz(int t) { return (((t >> 1) & 1) << 2) | ((t >> 2) & 3); }

// partial element e = ((dt*2 + nb)*16 + reg)*64 + lane holds C^T[d][r] with
// r = 32 nb + (lane & 31), d = 32 dt + 8 (reg >> 2) + 4 (lane >> 5) + (reg & 3).
//
// Per 128-token sub-tile: wave w projects its 32 tokens (K~^T = P_k k_norm^T,
// lane = token, so a rotation pair sits in one lane), applies silu and the
// rotation and writes K~ as bf16 hi + lo to LDS; after a barrier wave w
// accumulates the 32 rows d = 32 w .. of C^T = V^T K~ over all 128 tokens.
__global__ __launch_bounds__(256, 2) void comp_state_kernel(StateArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t vt[kSub * kVRow];        // V rows (swz_v)
  __shared__ __attribute__((aligned(16))) uint8_t kth[kSub * kRank * 2];   // K~ hi
  __shared__ __attribute__((aligned(16))) uint8_t ktl[kSub * kRank * 2];   // K~ lo
  // P_k rows (r, 256 bytes each); 16-byte chunk c of row r at slot c ^ (r & 15)
  __shared__ __attribute__((aligned(16))) uint8_t pks[kRank * kHeadDim * 2];
  const int bh = blockIdx.x, chunk = blockIdx.y;  // heads vary fastest: rope rows shared in L2
  const int b = bh / a.H, h = bh - b * a.H;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int g = lane >> 5, l32 = lane & 31;
  // tokens [t_begin, t_end): sub-chunk `sub` of causal chunk `cc`
  const int cc = chunk / a.nsub, sub = chunk - cc * a.nsub;
  const int t_begin = cc * a.span + sub * kChunk;
  const int t_end = min(min(t_begin + kChunk, (cc + 1) * a.span), a.N);

  // resources end at t_end: rows past it (the next chunk, or past N) read
  // zero and so add nothing to the state
  const uint32_t kst = (uint32_t)a.kns.n * 2, vst = (uint32_t)a.vs.n * 2;
  const uint32_t rows = (uint32_t)max(t_end, 1);
  const auto kr = make_rsrc(a.kn + b * a.kns.b + h * a.kns.h, (rows - 1) * kst + 256u);
  const auto vr = make_rsrc(a.v + b * a.vs.b + h * a.vs.h, (rows - 1) * vst + 256u);
  const auto rr = make_rsrc(a.rope, (uint32_t)a.N * kRopeBytes);

  // k_norm as B operand of P_k k_norm^T (token tw + l32, channels
  // 16 ks + 8 g .. +7) and the sub-tile's V rows (thread t moves chunks
  // e = t + 256 m -> row e/16, chunk e%16); rows past N read zero
  bf16x8 kf[8];
  u32x4 vrow[8];
  auto load_kv = [&](int t0, bf16x8 (&kd)[8], u32x4 (&vd)[8]) {
    const int tw = t0 + 32 * wave;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      kd[ks] = as_bf16x8(buf_ld16(kr, (uint32_t)(tw + l32) * kst + (16 * ks + 8 * g) * 2));
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int e = t + 256 * m, row = e >> 4, ch = e & 15;
      vd[m] = buf_ld16(vr, (uint32_t)(t0 + row) * vst + ch * 16);
    }
  };
  if (t_begin < t_end) load_kv(t_begin, kf, vrow);

  // P_k of this head into LDS
  const uint16_t* pkh = a.pk + (int64_t)h * kStateElems;
#pragma unroll
  for (int m = 0; m < kRank * 16 / 256; ++m) {
    const int e = t + 256 * m, r = e >> 4, c = e & 15;
    *reinterpret_cast<u32x4*>(pks + r * 256 + ((c ^ (r & 15)) << 4)) = ld16(pkh + 8 * e);
  }

  f32x16 acc[2];  // C^T rows d = 32 wave .., columns r = 32 nb + l32
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[nb][r] = 0.f;

  for (int t0 = t_begin; t0 < t_end; t0 += kSub) {
    const int tok = t0 + 32 * wave + l32;  // this lane's token in the projection
    // (cos, sin) of this lane's pairs m = 16 nb + 4 j + 2 g + {0, 1} at its
    // token: 16 contiguous bytes per (nb, j); issued before the next
    // sub-tile's loads, so waiting for them does not wait for those
    f32x4 csn[2][4];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        csn[nb][j] = __builtin_bit_cast(
            f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       rr, (uint32_t)tok * kRopeBytes + (uint32_t)(16 * nb + 4 * j + 2 * g) * 8u,
                       0, 0));
    __syncthreads();  // every wave is done reading the previous sub-tile's V and K~
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const int e = t + 256 * m, row = e >> 4, ch = e & 15;
      *reinterpret_cast<u32x4*>(vt + row * kVRow + swz_v(row, ch) * 16) = vrow[m];
    }
    // projection K~^T = P_k k_norm^T: lane holds token `tok`, rank indices
    // 32 nb + 8 j + 4 g + rr (register 4 j + rr)
    const int ln = fresh_lane(), fl32 = ln & 31, fg = ln >> 5;
    f32x16 pr[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) pr[nb][r] = 0.f;
      const int prow = fl32 + 32 * nb;
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        const bf16x8 pf = as_bf16x8(*reinterpret_cast<const u32x4*>(
            pks + prow * 256 + (((2 * ks + fg) ^ (prow & 15)) << 4)));
        pr[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf, kf[ks], pr[nb], 0, 0, 0);
      }
    }
    // the next sub-tile's k_norm and V (on the last sub-tile the current
    // one's again: the loads are issued on every path)
    load_kv(t0 + kSub < t_end ? t0 + kSub : t0, kf, vrow);
    // silu, rotation of pairs (rr 0, 1) and (2, 3), K~ split hi + lo into LDS
    const int trow = 32 * wave + fl32;  // this lane's token row in the sub-tile
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const f32x4 cj = csn[nb][j];
        float y[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) y[u] = silu(pr[nb][4 * j + u]);
        const float rv[4] = {fmaf(y[0], cj[0], -y[1] * cj[1]), fmaf(y[0], cj[1], y[1] * cj[0]),
                             fmaf(y[2], cj[2], -y[3] * cj[3]), fmaf(y[2], cj[3], y[3] * cj[2])};
        u32x2 wh, wl;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const u32x2 hl = split_pair(rv[2 * u], rv[2 * u + 1]);
          wh[u] = hl[0];
          wl[u] = hl[1];
        }
        // r = 32 nb + 8 j + 4 g .. +3: bytes 64 nb + 16 j + 8 g of the row
        const int c = 4 * nb + j;
        const int off = trow * 128 + ((c ^ kt_swz(trow)) << 4) + 8 * fg;
        *reinterpret_cast<u32x2*>(kth + off) = wh;
        *reinterpret_cast<u32x2*>(ktl + off) = wl;
      }
    __syncthreads();  // the sub-tile's V rows and K~ are in LDS

    // C^T[32 wave ..][.] += V^T K~ over the 128 tokens: A = V^T (channels
    // 32 wave + l32) and B = K~ (columns r), both by transposed reads whose
    // lane 16 G + 4 e + q reads row (token) r16 + 8 hf + 4 (G >> 1) + e
    {
      const int ln2 = fresh_lane();
      const int G = ln2 >> 4, e4 = (ln2 >> 2) & 3, q4 = ln2 & 3;
#pragma unroll
      for (int r16 = 0; r16 < kSub; r16 += 16) {
        u32x4 va, kh2[2], kl2[2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int row = r16 + 8 * hf + 4 * (G >> 1) + e4;
          // V^T: channels 32 wave + 16 (G & 1) + 4 q .. +3
          const int lc = 4 * wave + 2 * (G & 1) + (q4 >> 1);
          const u32x2 v2 = __builtin_bit_cast(
              u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                         (__attribute__((address_space(3))) i16x4*)(vt + row * kVRow +
                                                                    swz_v(row, lc) * 16 +
                                                                    (q4 & 1) * 8)));
          va[2 * hf] = v2[0];
          va[2 * hf + 1] = v2[1];
#pragma unroll
          for (int nb = 0; nb < 2; ++nb) {
            // K~: r = 32 nb + 16 (G & 1) + 4 q .. +3 -> chunk 4 nb + 2 (G & 1) + q / 2
            const int c = 4 * nb + 2 * (G & 1) + (q4 >> 1);
            const int off = row * 128 + ((c ^ kt_swz(row)) << 4) + (q4 & 1) * 8;
            const u32x2 h2 = __builtin_bit_cast(
                u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                           (__attribute__((address_space(3))) i16x4*)(kth + off)));
            const u32x2 l2 = __builtin_bit_cast(
                u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                           (__attribute__((address_space(3))) i16x4*)(ktl + off)));
            kh2[nb][2 * hf] = h2[0];
            kh2[nb][2 * hf + 1] = h2[1];
            kl2[nb][2 * hf] = l2[0];
            kl2[nb][2 * hf + 1] = l2[1];
          }
        }
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
          acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(va), as_bf16x8(kh2[nb]),
                                                            acc[nb], 0, 0, 0);
          acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(va), as_bf16x8(kl2[nb]),
                                                            acc[nb], 0, 0, 0);
        }
      }
    }
  }

  // this wave's rows of the chunk's partial C^T
  float* out = a.partial + ((int64_t)bh * a.nc * a.nsub + chunk) * kStateElems;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int r = 0; r < 16; ++r) out[((wave * 2 + nb) * 16 + r) * 64 + lane] = acc[nb][r];
}

// C^T[bh][c][d][r] of causal chunk c = sum over the chunks c2 of its window
// [c - window + 1, c] (all up to c for window 0), in ascending order, of
// T_c2 = the sum of c2's sub-chunk partials in order.  Without a window there
// is one chunk.  Each workgroup sums 256 of a head's elements, for every c.
__global__ __launch_bounds__(256) void comp_reduce_kernel(const float* __restrict__ partial,
                                                          int nc, int nsub, int window,
                                                          float* __restrict__ state) {
  const int bh = blockIdx.x;
  const int e = blockIdx.y * 256 + threadIdx.x;
  const float* src = partial + (int64_t)bh * nc * nsub * kStateElems + e;
  const int lane = e & 63, reg = (e >> 6) & 15, blk = e >> 10;  // blk = dt * 2 + nb
  const int dt = blk >> 1, nb = blk & 1;
  const int r = 32 * nb + (lane & 31);
  const int d = 32 * dt + 8 * (reg >> 2) + 4 * (lane >> 5) + (reg & 3);
  float* dst = state + (int64_t)bh * nc * kStateElems + d * kRank + r;
  auto chunk_sum = [&](int c2) {
    float t = 0.f;
    for (int u = 0; u < nsub; ++u) t += src[((int64_t)c2 * nsub + u) * kStateElems];
    return t;
  };
  if (window == 0) {  // running prefix: the same additions as the direct sums
    float s = 0.f;
    for (int c = 0; c < nc; ++c) {
      s += chunk_sum(c);
      dst[(int64_t)c * kStateElems] = s;
    }
  } else {
    for (int c = 0; c < nc; ++c) {
      float s = 0.f;
      for (int c2 = max(0, c - window + 1); c2 <= c; ++c2) s += chunk_sum(c2);
      dst[(int64_t)c * kStateElems] = s;
    }
  }
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
  int span;  // tokens per causal chunk (N without a window)
  int ntg;   // workgroups per causal chunk, ceil(span / (kOutTiles * 128))
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
  // tokens [t_beg, t_end) of causal chunk cc (one chunk without a window),
  // all of them using that chunk's state, in tiles of 128
  const int cc = blockIdx.y / a.ntg, grp = blockIdx.y - cc * a.ntg;
  const int c_end = min((cc + 1) * a.span, a.N);
  const int t_beg = cc * a.span + grp * kOutTiles * kSub;
  const int t_end = min(t_beg + kOutTiles * kSub, c_end);
  if (t_beg >= t_end) return;  // uniform: a short last chunk
  const int ntile = (t_end - t_beg + kSub - 1) / kSub;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int g = lane >> 5, l32 = lane & 31;

  // the first tile's per-token loads are issued first, so their latency
  // overlaps the staging of C^T and P_q
  bf16x8 qf[8];
  u32x2 osw[4][4];
  float gv;
  load_tok(a, b, h, min(t_beg + 32 * wave + l32, a.N - 1), g, qf, osw, gv);

  // C^T of this head and chunk as bf16 hi + lo into LDS: thread t converts
  // quads of 4 consecutive r (16-byte loads) and stores each as 8 bytes at
  // its permuted position
  const int nc = (a.N + a.span - 1) / a.span;
  const float* st = a.state + ((int64_t)bh * nc + cc) * kStateElems;
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

  for (int tile = 0; tile < ntile; ++tile) {
    const int tok = t_beg + tile * kSub + 32 * wave + l32;  // this lane's token
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
    load_tok(a, b, h, min(tile + 1 < ntile ? tok + kSub : tok, a.N - 1), g, qn, on, gn);

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
    u32x4 qtw[4], qlw[4];  // packed bf16 pairs
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
        for (int u = 0; u < 2; ++u) {
          const u32x2 hl = split_pair(rv[2 * u], rv[2 * u + 1]);
          qtw[s2][half / 2 + u] = hl[0];
          qlw[s2][half / 2 + u] = hl[1];
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
        y[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cl, as_bf16x8(qtw[s2]), y[dt], 0, 0, 0);
        y[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cf, as_bf16x8(qlw[s2]), y[dt], 0, 0, 0);
        y[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(cf, as_bf16x8(qtw[s2]), y[dt], 0, 0, 0);
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
    // sums of squares in four independent partials each (short dependency
    // chains)
    float py[4] = {0.f, 0.f, 0.f, 0.f}, po[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const u32x2 w = osw[dt][j];
        const float o4[4] = {bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          py[u] = fmaf(y[dt][4 * j + u], y[dt][4 * j + u], py[u]);
          po[u] = fmaf(o4[u], o4[u], po[u]);
        }
      }
    float ss_y = (py[0] + py[1]) + (py[2] + py[3]);
    float ss_o = (po[0] + po[1]) + (po[2] + po[3]);
    ss_y += __shfl_xor(ss_y, 32, kWave);
    ss_o += __shfl_xor(ss_o, 32, kWave);
    const float rstd = 1.f / sqrtf(ss_y * (1.f / kHeadDim) + a.eps);
    const float rms_o = sqrtf(ss_o * (1.f / kHeadDim));
    const float coef = gv * rms_o * rstd;
    if (tok < t_end) {
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
            wo[2 * jj] = cvt_pk_bf16(x[0], x[1]);
            wo[2 * jj + 1] = cvt_pk_bf16(x[2], x[3]);
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

// Tokens per causal chunk (the whole sequence without a window) and the
// number of chunks, which is the number of states per head.
static int comp_span(const Shape& s) {
  return s.causal_chunk > 0 ? std::min(s.causal_chunk, s.N) : s.N;
}
int comp_state_chunks(const Shape& s) { return (s.N + comp_span(s) - 1) / comp_span(s); }

size_t comp_state_workspace_bytes(const Shape& s) {
  const int64_t nsub = (comp_span(s) + kChunk - 1) / kChunk;
  return (size_t)s.B * s.H * comp_state_chunks(s) * nsub * kStateElems * sizeof(float);
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
  a.span = comp_span(s);
  a.nc = comp_state_chunks(s);
  a.nsub = (a.span + kChunk - 1) / kChunk;
  comp_state_kernel<<<dim3(s.B * s.H, a.nc * a.nsub), 256, 0, stream>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  comp_reduce_kernel<<<dim3(s.B * s.H, kReduceSplit), 256, 0, stream>>>(
      a.partial, a.nc, a.nsub, s.causal_chunk > 0 ? s.causal_window : 0, state);
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
  a.span = comp_span(s);
  a.ntg = (a.span + kOutTiles * kSub - 1) / (kOutTiles * kSub);
  comp_out_kernel<<<dim3(s.B * s.H, comp_state_chunks(s) * a.ntg), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace sa

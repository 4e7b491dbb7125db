// W8A8 FP8 (OCP e4m3) linear layer on gfx950 (paper §4.3): activations are
// quantised per token at run time in one pass over memory, weights per output
// channel once offline (the same row rule), and the product
//   y[m][n] = (sum_k xq[m][k] * wq[n][k]) * sx[m] * sw[n] + bias[n]
// runs on the fp8 matrix cores with fp32 accumulation and a bf16 output.
//
// Row quantisation: one wavefront per row, the whole row held in registers
// (16-byte chunks), the absolute maximum reduced with integer compares on the
// bf16 magnitude bits; a = max(amax, 2^-100), scale = a / 448 and
// codes = e4m3(x * (448 / a)), each quotient and product a correctly rounded
// fp32 operation, the code rounded to nearest with ties to even.
//
// Product: persistent workgroups (4 waves, one per CU) walk 256 x 256 output
// tiles, each computed transposed (D^T = W X^T), so that each lane ends with
// four consecutive output channels of one token; the tile leaves through LDS
// as whole row segments.  Each wave owns a 128 x 128 quarter: 4 x 4
// accumulators of v_mfma_scale_f32_32x32x64_f8f6f4 (unit scales).  K
// advances 128 bytes per stage, so that every row segment a stage copies is
// one whole 128-byte line (64-byte segments halve the L2 -> LDS rate); a
// stage (the tile's 256 weight rows and 256 activation rows, 64 KB) moves
// global -> LDS with buffer_load ... lds, issued from inline asm, rows past
// M or N reading zero.  Two stage buffers: the copy of stage s+2 is issued
// at the barrier that releases stage s, between stage s's two MFMA steps,
// so it has a whole stage of MFMAs to land; the copy pipeline runs on across
// tile boundaries.  Tiles are ordered in groups of `group_m` tile rows and
// dealt to the 8 XCDs in contiguous runs, so the workgroups that run
// together on one XCD share their activation and weight rows in its L2.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

// Two fp32 values as packed bf16, rounded to nearest even by the hardware
// conversion (v_cvt_pk_bf16_f32): one instruction per pair.
__device__ __forceinline__ uint32_t cvt_pk_bf16(float lo, float hi) {
  typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
  const bf16x2_t t = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, t);
}

// ---- per-row quantisation --------------------------------------------------

constexpr int kRowsPerGroup = 4;  // one row per wave

template <int P>  // 16-byte chunks per lane: rows of up to 512 * P elements
__global__ __launch_bounds__(256) void quant_rows_kernel(const uint16_t* __restrict__ x,
                                                         int64_t ldx, int64_t rows, int cols,
                                                         uint8_t* __restrict__ q,
                                                         float* __restrict__ scale) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerGroup + wave;
  if (row >= rows) return;  // whole wave; no barrier below
  const uint16_t* src = x + row * ldx;
  const int nch = cols >> 3;

  u32x4 v[P];
  uint32_t amax = 0;  // bf16 magnitude bits: integer order is value order
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int c = lane + kWave * p;
    if (c < nch) {
      v[p] = ld16(src + 8 * c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        amax = max(amax, v[p][e] & 0x7fffu);
        amax = max(amax, (v[p][e] >> 16) & 0x7fffu);
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, o, kWave));
  const float a = fmaxf(__uint_as_float(amax << 16), 0x1p-100f);
  const float inv = __fdiv_rn(448.f, a);
  if (lane == 0) scale[row] = __fdiv_rn(a, 448.f);

  uint8_t* dst = q + row * (int64_t)cols;
#pragma unroll
  for (int p = 0; p < P; ++p) {
    const int c = lane + kWave * p;
    if (c < nch) {
      u32x2 out;
#pragma unroll
      for (int hw = 0; hw < 2; ++hw) {
        const uint32_t w0 = v[p][2 * hw], w1 = v[p][2 * hw + 1];
        out[hw] = e4m3_rne(bf16_lo(w0) * inv) | (e4m3_rne(bf16_hi(w0) * inv) << 8) |
                  (e4m3_rne(bf16_lo(w1) * inv) << 16) | (e4m3_rne(bf16_hi(w1) * inv) << 24);
      }
      *reinterpret_cast<u32x2*>(dst + 8 * c) = out;
    }
  }
}

// Rows longer than the register-resident variants: the same arithmetic over
// two passes (the second re-reads the row, mostly from L2).
__global__ __launch_bounds__(256) void quant_rows_stream_kernel(const uint16_t* __restrict__ x,
                                                                int64_t ldx, int64_t rows,
                                                                int cols, uint8_t* __restrict__ q,
                                                                float* __restrict__ scale) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * kRowsPerGroup + wave;
  if (row >= rows) return;
  const uint16_t* src = x + row * ldx;
  const int nch = cols >> 3;
  uint32_t amax = 0;
  for (int c = lane; c < nch; c += kWave) {
    const u32x4 v = ld16(src + 8 * c);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      amax = max(amax, v[e] & 0x7fffu);
      amax = max(amax, (v[e] >> 16) & 0x7fffu);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, o, kWave));
  const float a = fmaxf(__uint_as_float(amax << 16), 0x1p-100f);
  const float inv = __fdiv_rn(448.f, a);
  if (lane == 0) scale[row] = __fdiv_rn(a, 448.f);
  uint8_t* dst = q + row * (int64_t)cols;
  for (int c = lane; c < nch; c += kWave) {
    const u32x4 v = ld16(src + 8 * c);
    u32x2 out;
#pragma unroll
    for (int hw = 0; hw < 2; ++hw) {
      const uint32_t w0 = v[2 * hw], w1 = v[2 * hw + 1];
      out[hw] = e4m3_rne(bf16_lo(w0) * inv) | (e4m3_rne(bf16_hi(w0) * inv) << 8) |
                (e4m3_rne(bf16_lo(w1) * inv) << 16) | (e4m3_rne(bf16_hi(w1) * inv) << 24);
    }
    *reinterpret_cast<u32x2*>(dst + 8 * c) = out;
  }
}

// ---- product ---------------------------------------------------------------

constexpr int kBM = 256;                       // tokens per tile
constexpr int kBN = 256;                       // output channels per tile
constexpr int kBK = 128;                       // bytes of K per stage: whole 128-byte lines
constexpr int kStages = 2;
constexpr int kHalfBytes = kBN * kBK;          // 32 KB: the weight (or activation) rows of a stage
constexpr int kStageBytes = 2 * kHalfBytes;    // [weights | activations]
constexpr int kOneE8m0 = 127;                  // E8M0 code of 1

// Physical 16-byte slot of logical chunk c (0..7) of a 128-byte row: the
// sixteen lanes that one LDS cycle serves read sixteen consecutive rows at
// the same logical chunk; row 2a + b then lands in 16-byte bank group
// 8b + (c ^ a) of the 256-byte bank window, all sixteen distinct.
__device__ __forceinline__ int swz128(int row, int c) { return c ^ ((row >> 1) & 7); }

__device__ __forceinline__ void wait_vm0() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x0F70);
}
__device__ __forceinline__ void wait_vm16() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x4F70);
}
__device__ __forceinline__ void wait_lgkm0() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0xC07F);
}

struct LinArgs {
  const uint8_t* x;   // activation codes [M][K], row stride ldx bytes
  const float* sx;    // [M]
  const uint8_t* w;   // weight codes [N][K], row stride ldw bytes
  const float* sw;    // [N]
  const float* bias;  // [N] or null
  uint16_t* y;        // bf16 [M][N], row stride ldy elements
  int64_t ldx, ldw, ldy;
  int M, N, K;
  int tiles_m, tiles_n, group_m;
};

constexpr int kOutLds = 4 * 4096;    // per wave: 32 rows x 64 output channels of bf16
constexpr int kScaleLds = 4 * 1024;  // sx | sw | bias of the current tile (+ one spare)
constexpr int kLdsBytes = kStages * kStageBytes + kOutLds + kScaleLds;

// Lane index within the wavefront, recomputed at every use (volatile asm of
// the two mbcnt instructions), so that no register holds it across a loop.
__device__ __forceinline__ int fresh_lane_id() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Tile t (in the grouped order) -> its first token and output channel.
__device__ __forceinline__ void tile_origin(const LinArgs& a, int t, int& m0, int& n0) {
  const int gsz = a.group_m * a.tiles_n;
  const int grp = t / gsz;
  const int first_m = grp * a.group_m;
  const int gm = min(a.group_m, a.tiles_m - first_m);
  const int within = t - grp * gsz;
  m0 = (first_m + within % gm) * kBM;
  n0 = (within / gm) * kBN;
}

// Global -> LDS copy of one stage (K slice `k0` of the tile's 256 weight rows
// and 256 activation rows) into the stage buffer at LDS byte address `base`.
__device__ __forceinline__ void copy_stage(uint32_t base, __amdgpu_buffer_rsrc_t wr,
                                           __amdgpu_buffer_rsrc_t xr, const uint32_t (&woff)[8],
                                           const uint32_t (&xoff)[8], uint32_t k0) {
#pragma unroll
  for (int i = 0; i < 8; ++i) dma16(base + 8 * i * kBK, wr, woff[i], k0);
#pragma unroll
  for (int i = 0; i < 8; ++i) dma16(base + kHalfBytes + 8 * i * kBK, xr, xoff[i], k0);
}

// A (weights) and B (activations) fragments of one 64-byte K step of the
// stage buffer `sb`: fa*/fb* are the byte offsets of the lane's two 16-byte
// chunks in the first A / B row of the step (swizzle applied).
__device__ __forceinline__ void read_frags(const uint8_t* sb, uint32_t fa0, uint32_t fa1,
                                           uint32_t fb0, uint32_t fb1, i32x8 (&fa)[4],
                                           i32x8 (&fb)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const u32x4 lo = *reinterpret_cast<const u32x4*>(sb + fa0 + 32 * i * kBK);
    const u32x4 hi = *reinterpret_cast<const u32x4*>(sb + fa1 + 32 * i * kBK);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      fa[i][e] = (int)lo[e];
      fa[i][4 + e] = (int)hi[e];
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const u32x4 lo = *reinterpret_cast<const u32x4*>(sb + fb0 + 32 * j * kBK);
    const u32x4 hi = *reinterpret_cast<const u32x4*>(sb + fb1 + 32 * j * kBK);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      fb[j][e] = (int)lo[e];
      fb[j][4 + e] = (int)hi[e];
    }
  }
}

// Part t (0..15) of the fragment reads of one K step: A fragments 0..3 then
// B fragments 0..3, two 16-byte halves each.
template <int T>
__device__ __forceinline__ void read_frag_part(const uint8_t* sb, const uint32_t (&fk)[4],
                                               i32x8 (&fa)[4], i32x8 (&fb)[4]) {
  constexpr int f = T >> 1, h = T & 1;
  if constexpr (f < 4) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(sb + fk[h] + 32 * f * kBK);
#pragma unroll
    for (int e = 0; e < 4; ++e) fa[f][4 * h + e] = (int)v[e];
  } else {
    const u32x4 v = *reinterpret_cast<const u32x4*>(sb + fk[2 + h] + 32 * (f - 4) * kBK);
#pragma unroll
    for (int e = 0; e < 4; ++e) fb[f - 4][4 * h + e] = (int)v[e];
  }
}

// MFMA t (0..15) of one K step: accumulator (i, j) = (t % 4, t / 4).
template <int T, bool FIRST>
__device__ __forceinline__ void mfma_one(f32x16 (&acc)[4][4], const i32x8 (&fa)[4],
                                         const i32x8 (&fb)[4]) {
  constexpr int i = T & 3, j = T >> 2;
  const f32x16 zero = {};
  acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
      fa[i], fb[j], FIRST ? zero : acc[i][j], 0, 0, 0, kOneE8m0, 0, kOneE8m0);
}

// The two interleaved phases of a stage, each one MFMA step with the reads
// and copies it hides: MFMA t, then fragment part t (and copy t).
template <int T, bool FIRST>
__device__ __forceinline__ void phase0(f32x16 (&acc)[4][4], const i32x8 (&fa0)[4],
                                       const i32x8 (&fb0)[4], const uint8_t* sb,
                                       const uint32_t (&fk1)[4], i32x8 (&fa1)[4],
                                       i32x8 (&fb1)[4]) {
  if constexpr (T < 16) {
    mfma_one<T, FIRST>(acc, fa0, fb0);
    read_frag_part<T>(sb, fk1, fa1, fb1);
    __builtin_amdgcn_sched_barrier(0);
    phase0<T + 1, FIRST>(acc, fa0, fb0, sb, fk1, fa1, fb1);
  }
}
template <int T>
__device__ __forceinline__ void phase1(f32x16 (&acc)[4][4], const i32x8 (&fa1)[4],
                                       const i32x8 (&fb1)[4], const uint8_t* nb,
                                       const uint32_t (&fk0)[4], i32x8 (&fa0)[4],
                                       i32x8 (&fb0)[4], uint32_t cbuf,
                                       __amdgpu_buffer_rsrc_t wr, __amdgpu_buffer_rsrc_t xr,
                                       const uint32_t (&woff)[8], const uint32_t (&xoff)[8],
                                       uint32_t k0) {
  if constexpr (T < 16) {
    if constexpr (T < 8)
      dma16(cbuf + 8 * T * kBK, wr, woff[T], k0);
    else
      dma16(cbuf + kHalfBytes + 8 * (T - 8) * kBK, xr, xoff[T - 8], k0);
    mfma_one<T, false>(acc, fa1, fb1);
    read_frag_part<T>(nb, fk0, fa0, fb0);
    __builtin_amdgcn_sched_barrier(0);
    phase1<T + 1>(acc, fa1, fb1, nb, fk0, fa0, fb0, cbuf, wr, xr, woff, xoff, k0);
  }
}

// Persistent: one workgroup per CU walks its share of the output tiles, and
// the copy pipeline runs on across tile boundaries (the first stages of the
// next tile are in flight while the current one finishes and is stored).
__global__ __launch_bounds__(256) void linear_w8a8_kernel(LinArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kLdsBytes];
  constexpr int kOutOff = kStages * kStageBytes;  // byte offsets in lds
  constexpr int kScaleOff = kOutOff + kOutLds;

  // Tiles of this workgroup.  Dispatch deals workgroup ids round-robin over
  // the 8 XCDs; XCD x owns a contiguous run of the grouped tile order, and its
  // workgroups take that run's tiles in turn, so the ones running together on
  // an XCD share activation and weight rows in its L2.
  const int T = a.tiles_m * a.tiles_n;
  const int G = gridDim.x;
  const int id = blockIdx.x, xcd = id & 7, lw = id >> 3;
  const int wgs_x = (G >> 3) + (xcd < (G & 7) ? 1 : 0);
  const int tiles_x = (T >> 3) + (xcd < (T & 7) ? 1 : 0);
  const int t_first = xcd * (T >> 3) + min(xcd, T & 7) + lw;
  const int ntiles = lw < tiles_x ? (tiles_x - lw + wgs_x - 1) / wgs_x : 0;
  if (ntiles == 0) return;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int wn = wv >> 1, wm = wv & 1;  // this wave's 128 x 128 quarter (uniform)
  const int g = lane >> 5, l32 = lane & 31;
  const int S = a.K / kBK;
  const uint32_t lds0 = lds_addr(lds);

  const uint32_t cbase = lds0 + (uint32_t)(64 * wv * kBK);  // this wave's rows in stage 0
  // Per-lane copy offsets and fragment addresses.  They are derived again at
  // every tile from a freshly computed lane index, so that they are not live
  // (and spilled) across the epilogue, where the accumulators need the
  // registers.
  uint32_t woff[8], xoff[8], fk[2][4];  // fk[ks] = {fa0, fa1, fb0, fb1} of K step ks
#define LIN_LANE_SETUP()                                                                      \
  do {                                                                                        \
    const int ln_ = fresh_lane_id();                                                          \
    /* copies: wave w moves rows 64w .. 64w+63 of both halves, 8 rows per instruction;        \
       lane l lands in slot l%8 of row l/8 (the swizzle is an involution) */                  \
    _Pragma("unroll") for (int i_ = 0; i_ < 8; ++i_) {                                        \
      const int row_ = 64 * wv + 8 * i_ + (ln_ >> 3);                                         \
      const int c_ = swz128(row_, ln_ & 7);                                                   \
      woff[i_] = (uint32_t)(row_ * a.ldw + 16 * c_);                                          \
      xoff[i_] = (uint32_t)(row_ * a.ldx + 16 * c_);                                          \
    }                                                                                         \
    /* fragments: A (weights) row 128 wn + 32 i + l32, B (activations) row 128 wm + 32 j +    \
       l32; K step ks, bytes 64 ks + 32 g .. + 31 = logical chunks 4 ks + 2 g, + 1; the       \
       swizzle term (row >> 1) & 7 depends on l32 only */                                     \
    const int g_ = ln_ >> 5, l_ = ln_ & 31, s1_ = (l_ >> 1) & 7;                              \
    _Pragma("unroll") for (int ks_ = 0; ks_ < 2; ++ks_) {                                     \
      const int c0_ = 4 * ks_ + 2 * g_;                                                       \
      fk[ks_][0] = (uint32_t)((128 * wn + l_) * kBK + 16 * (c0_ ^ s1_));                      \
      fk[ks_][1] = (uint32_t)((128 * wn + l_) * kBK + 16 * ((c0_ + 1) ^ s1_));                \
      fk[ks_][2] = (uint32_t)(kHalfBytes + (128 * wm + l_) * kBK + 16 * (c0_ ^ s1_));         \
      fk[ks_][3] = (uint32_t)(kHalfBytes + (128 * wm + l_) * kBK + 16 * ((c0_ + 1) ^ s1_));   \
    }                                                                                         \
  } while (0)
  LIN_LANE_SETUP();


  // current and next tile: origins and the byte ranges of their rows
  int tile = t_first, m0, n0, nm0, nn0;
  tile_origin(a, tile, m0, n0);
  bool has_next = ntiles > 1;
  nm0 = m0;
  nn0 = n0;
  if (has_next) tile_origin(a, tile + wgs_x, nm0, nn0);
  auto wbytes = [&](int n) { return (uint32_t)(min(kBN, a.N - n) * a.ldw); };
  auto xbytes = [&](int m) { return (uint32_t)(min(kBM, a.M - m) * a.ldx); };

  // Copy number q of the current tile (q >= S: stage q - S of the next one,
  // which needs S >= 2; past the end a repeat of the last stage, into a
  // buffer that is never read again): every stage issues the same 16 copies
  // per wave.
#define LIN_COPY(q, buf)                                                                      \
  do {                                                                                        \
    const bool cur_ = (q) < S;                                                                \
    const bool use_c_ = cur_ || !has_next;                                                    \
    const int st_ = cur_ ? (q) : (has_next ? (q) - S : S - 1);                               \
    const int mo_ = use_c_ ? m0 : nm0, no_ = use_c_ ? n0 : nn0;                               \
    copy_stage(cbase + (uint32_t)((buf) * kStageBytes),                                       \
               make_rsrc(a.w + (int64_t)no_ * a.ldw, wbytes(no_)),                            \
               make_rsrc(a.x + (int64_t)mo_ * a.ldx, xbytes(mo_)), woff, xoff,                \
               (uint32_t)(st_ * kBK));                                                        \
  } while (0)

  // scale vectors of the current tile into LDS: wave 0 sx, wave 1 sw, wave 2
  // bias (zeros without bias: an empty range reads zero), wave 3 a spare copy
  // of sx; 1 KB each
#define LIN_COPY_SCALES()                                                                     \
  do {                                                                                        \
    const int which_ = wv == 3 ? 0 : wv;                                                      \
    const float* src_ = which_ == 0 ? a.sx + m0 : (which_ == 1 ? a.sw + n0 : a.bias + n0);   \
    const int valid_ = which_ == 0 ? min(kBM, a.M - m0)                                       \
                                   : (which_ == 2 && !a.bias ? 0 : min(kBN, a.N - n0));       \
    dma16(lds0 + (uint32_t)kScaleOff + 1024u * wv,                                            \
          make_rsrc(which_ == 2 && !a.bias ? a.sw : src_, (uint32_t)valid_ * 4u),             \
          16u * (uint32_t)fresh_lane_id(),                                                    \
          0u);                                                                                \
  } while (0)

  f32x16 acc[4][4];
  i32x8 fa0[4], fb0[4], fa1[4], fb1[4];  // fragments of K steps 0 and 1 of a stage

  // prologue: stages 0 and 1 of the sequence, the first tile's scales
  LIN_COPY(0, 0);
  LIN_COPY(1, 1);
  LIN_COPY_SCALES();
  wait_vm16();  // stage 0 landed (this wave's part); stage 1 and the scales may be in flight
  barrier_keep_loads();
  read_frags(lds, fk[0][0], fk[0][1], fk[0][2], fk[0][3], fa0, fb0);
  int j = 0;  // global stage number: stage s of the k-th tile is k S + s, in buffer j % 2

  // One stage (K = 128 bytes, two MFMA steps), starting with the fragments
  // of its first step in registers.  Phase 0: the first step's 16 MFMAs,
  // each followed by one part of the second step's fragment reads.  Then the
  // wait for the next stage and the barrier that releases this one's buffer.
  // Phase 1: the second step's MFMAs, each preceded by one of the 16 copies
  // of the stage two ahead (into the released buffer) and followed by one
  // part of the next stage's first-step fragments.  Spreading the copies
  // keeps the texture addresser's queue short, so the wave never blocks on a
  // copy while the matrix cores idle.
#define LIN_STAGE(s, FIRST)                                                                   \
  do {                                                                                        \
    phase0<0, FIRST>(acc, fa0, fb0, lds + (j & 1) * kStageBytes, fk[1], fa1, fb1);            \
    wait_vm0();                                                                               \
    wait_lgkm0();                                                                             \
    barrier_keep_loads();                                                                     \
    const int q_ = (s) + kStages;                                                             \
    const bool cur_ = q_ < S;                                                                 \
    const bool use_c_ = cur_ || !has_next;                                                    \
    const int st_ = cur_ ? q_ : (has_next ? q_ - S : S - 1);                                  \
    const int mo_ = use_c_ ? m0 : nm0, no_ = use_c_ ? n0 : nn0;                               \
    phase1<0>(acc, fa1, fb1, lds + ((j + 1) & 1) * kStageBytes, fk[0], fa0, fb0,              \
              cbase + (uint32_t)((j & 1) * kStageBytes),                                      \
              make_rsrc(a.w + (int64_t)no_ * a.ldw, wbytes(no_)),                             \
              make_rsrc(a.x + (int64_t)mo_ * a.ldx, xbytes(mo_)), woff, xoff,                 \
              (uint32_t)(st_ * kBK));                                                         \
    ++j;                                                                                      \
  } while (0)

  for (int k = 0; k < ntiles; ++k) {
    LIN_LANE_SETUP();
    LIN_STAGE(0, true);
    for (int s = 1; s < S; ++s) LIN_STAGE(s, false);

    // (The scale vectors of this tile were copied before its first stage,
    // whose wait and barrier have covered them.)
    // Epilogue through LDS in 8 passes of 32 tokens x 64 output channels per
    // wave, each stored as 128-byte row segments.  acc[i][jj][4q + u] is
    // output channel 128 wn + 32 i + 8 q + 4 g + u of token 128 wm + 32 jj +
    // l32 (tile-local).  Staging row r holds 64 channels (8 chunks of 16
    // bytes, chunk c at slot c ^ (r & 7)).
    // (a freshly computed lane index, so that the compiler derives the
    // epilogue addresses here instead of keeping them live across the main
    // loop)
    const int le = fresh_lane_id();
    const int ge = le >> 5, l32e = le & 31;
    uint8_t* stg = lds + kOutOff + wv * 4096;
    const float* sxl = reinterpret_cast<const float*>(lds + kScaleOff);
    const float* swl = sxl + 256;
    const float* bl = sxl + 512;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const float sxv = sxl[128 * wm + 32 * jj + l32e];
#pragma unroll
      for (int ih = 0; ih < 2; ++ih) {
        __builtin_amdgcn_sched_barrier(0);  // one pass at a time: bounded registers
#pragma unroll
        for (int i2 = 0; i2 < 2; ++i2) {
          const int i = 2 * ih + i2;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int nl = 128 * wn + 32 * i + 8 * q + 4 * ge;
            const f32x4 swv = *reinterpret_cast<const f32x4*>(swl + nl);
            const f32x4 bv = *reinterpret_cast<const f32x4*>(bl + nl);
            float v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) v[u] = fmaf(acc[i][jj][4 * q + u] * sxv, swv[u], bv[u]);
            u32x2 o;
            o[0] = cvt_pk_bf16(v[0], v[1]);
            o[1] = cvt_pk_bf16(v[2], v[3]);
            const int c = 4 * i2 + q;  // chunk of 8 channels within the 64
            *reinterpret_cast<u32x2*>(stg + l32e * 128 + ((c ^ (l32e & 7)) << 4) + 8 * ge) = o;
          }
        }
        wait_lgkm0();  // the wave reads back only what it wrote itself
        const int c = le & 7;
        const int n = n0 + 128 * wn + 64 * ih + 8 * c;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          const int r = 8 * p + (le >> 3);
          const u32x4 v = *reinterpret_cast<const u32x4*>(stg + r * 128 + ((c ^ (r & 7)) << 4));
          const int m = m0 + 128 * wm + 32 * jj + r;
          if (m < a.M && n < a.N) st16(a.y + (int64_t)m * a.ldy + n, v);
        }
        wait_lgkm0();  // reads done before the next pass overwrites the staging rows
      }
    }

    // advance: the next tile becomes current; the copies of its first stages
    // are already in flight
    tile += wgs_x;
    m0 = nm0;
    n0 = nn0;
    has_next = k + 2 < ntiles;
    if (has_next) tile_origin(a, tile + wgs_x, nm0, nn0);
    if (k + 1 < ntiles) {
      // the scale vectors of the next tile: every wave has read this tile's
      // (its epilogue waited for its LDS reads); the barrier covers them all
      barrier_keep_loads();
      LIN_COPY_SCALES();
    }
  }
#undef LIN_STAGE
#undef LIN_LANE_SETUP
#undef LIN_COPY_SCALES
#undef LIN_COPY
  wait_vm0();  // the repeated copies past the end
}

}  // namespace

hipError_t launch_quant_rows_fp8(const void* x, int64_t ldx, int64_t rows, int cols, uint8_t* q,
                                 float* scale, hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + kRowsPerGroup - 1) / kRowsPerGroup));
  const uint16_t* xp = static_cast<const uint16_t*>(x);
  const int nch = cols / 8;
  if (nch <= 64 * 4)
    quant_rows_kernel<4><<<grid, 256, 0, stream>>>(xp, ldx, rows, cols, q, scale);
  else if (nch <= 64 * 10)
    quant_rows_kernel<10><<<grid, 256, 0, stream>>>(xp, ldx, rows, cols, q, scale);
  else if (nch <= 64 * 16)
    quant_rows_kernel<16><<<grid, 256, 0, stream>>>(xp, ldx, rows, cols, q, scale);
  else if (nch <= 64 * 28)
    quant_rows_kernel<28><<<grid, 256, 0, stream>>>(xp, ldx, rows, cols, q, scale);
  else
    quant_rows_stream_kernel<<<grid, 256, 0, stream>>>(xp, ldx, rows, cols, q, scale);
  return hipGetLastError();
}

hipError_t launch_linear_w8a8(const LinearIn& in, hipStream_t stream) {
  if (in.M == 0 || in.N == 0) return hipSuccess;
  LinArgs a{};
  a.x = in.xq;
  a.sx = in.sx;
  a.w = in.wq;
  a.sw = in.sw;
  a.bias = in.bias;
  a.y = static_cast<uint16_t*>(in.y);
  a.ldx = in.ldx;
  a.ldw = in.ldw;
  a.ldy = in.ldy;
  a.M = (int)in.M;
  a.N = (int)in.N;
  a.K = (int)in.K;
  a.tiles_m = (int)((in.M + kBM - 1) / kBM);
  a.tiles_n = (int)((in.N + kBN - 1) / kBN);
  a.group_m = in.group_m > 0 ? in.group_m : 4;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  const int64_t T = (int64_t)a.tiles_m * a.tiles_n;
  const int grid = (int)(T < cus ? T : cus);  // one persistent workgroup per CU
  linear_w8a8_kernel<<<dim3((unsigned)grid), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace sa

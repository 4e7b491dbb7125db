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
// Product: one workgroup (4 waves) per 256 x 256 output tile, computed
// transposed (D^T = W X^T), so that each lane ends with four consecutive
// output channels of one token; the tile leaves through LDS as whole
// 256-byte row segments.  Each wave owns a 128 x 128
// quarter: 4 x 4 accumulators of v_mfma_scale_f32_32x32x64_f8f6f4 (unit
// scales).  K advances 64 bytes per stage; a stage is the 256 weight rows and
// 256 activation rows of that K slice (32 KB), moved global -> LDS with
// buffer_load ... lds (issued from inline asm, rows past M or N read zero),
// four stages in flight (128 KB).  Each stage is read once per wave as
// fragments; the barrier that releases a stage's buffer sits between the two
// halves of the previous stage's MFMAs, so the next fragments load while the
// matrix cores still work.  Tiles are ordered in groups of `group_m` tile
// rows and dealt to the 8 XCDs in contiguous runs, so the workgroups that run
// together on one XCD share their activation and weight rows in its L2.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

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
constexpr int kBK = 64;                        // bytes of K per stage
constexpr int kStages = 4;
constexpr int kHalfBytes = kBN * kBK;          // 16 KB: the weight (or activation) rows of a stage
constexpr int kStageBytes = 2 * kHalfBytes;    // [weights | activations]
constexpr int kOneE8m0 = 127;                  // E8M0 code of 1

// Physical 16-byte slot of logical chunk c (0..3) of a 64-byte row: the
// sixteen lanes that one LDS cycle serves read sixteen consecutive rows at
// the same logical chunk; row 4a + b then lands in 16-byte bank group
// 4b + (c ^ a) of the 256-byte bank window, all sixteen distinct.
__device__ __forceinline__ int swz64(int row, int c) { return c ^ ((row >> 2) & 3); }

__device__ __forceinline__ void wait_vm0() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x0F70);
}
__device__ __forceinline__ void wait_vm8() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x0F78);
}
__device__ __forceinline__ void wait_vm16() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x4F70);
}
__device__ __forceinline__ void wait_vm24() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x4F78);
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

__global__ __launch_bounds__(256) void linear_w8a8_kernel(LinArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kStages * kStageBytes];

  // tile of this workgroup: contiguous runs per XCD (dispatch deals
  // workgroup ids round-robin over the 8 XCDs), grouped order inside
  const int T = a.tiles_m * a.tiles_n;
  const int id = blockIdx.x, xcd = id & 7, local = id >> 3;
  const int per = T >> 3, rem = T & 7;
  const int t = xcd * per + min(xcd, rem) + local;
  const int gsz = a.group_m * a.tiles_n;
  const int grp = t / gsz;
  const int first_m = grp * a.group_m;
  const int gm = min(a.group_m, a.tiles_m - first_m);
  const int within = t - grp * gsz;
  const int m0 = (first_m + within % gm) * kBM;
  const int n0 = (within / gm) * kBN;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const int wn = wave >> 1, wm = wave & 1;  // this wave's 128 x 128 quarter
  const int g = lane >> 5, l32 = lane & 31;

  // copies: wave w moves rows 64w .. 64w+63 of both halves, 16 rows per
  // instruction; lane l lands in slot l%4 of row l/4
  const auto wr = make_rsrc(a.w + (int64_t)n0 * a.ldw, (uint32_t)(min(kBN, a.N - n0) * a.ldw));
  const auto xr = make_rsrc(a.x + (int64_t)m0 * a.ldx, (uint32_t)(min(kBM, a.M - m0) * a.ldx));
  uint32_t woff[4], xoff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 64 * wave + 16 * i + (lane >> 2);
    const int c = swz64(row, lane & 3);  // logical chunk stored in this slot (the map is an involution)
    woff[i] = (uint32_t)(row * a.ldw + 16 * c);
    xoff[i] = (uint32_t)(row * a.ldx + 16 * c);
  }
  const uint32_t lds0 = lds_addr(lds);
  auto copy_stage = [&](int st, int buf) {
    const uint32_t base = lds0 + (uint32_t)(buf * kStageBytes + 64 * wv * kBK);
    const uint32_t k0 = (uint32_t)(st * kBK);
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16(base + 16 * i * kBK, wr, woff[i], k0);
#pragma unroll
    for (int i = 0; i < 4; ++i) dma16(base + kHalfBytes + 16 * i * kBK, xr, xoff[i], k0);
  };

  // fragment addresses: A (weights) row 128 wn + 32 i + l32, B (activations)
  // row 128 wm + 32 j + l32; bytes 32 g .. 32 g + 31 of the row = logical
  // chunks 2g, 2g + 1.  The swizzle term (row >> 2) & 3 depends on l32 only.
  const int s1 = (l32 >> 2) & 3;
  const uint32_t fa0 = (uint32_t)((128 * wn + l32) * kBK + 16 * ((2 * g) ^ s1));
  const uint32_t fa1 = (uint32_t)((128 * wn + l32) * kBK + 16 * ((2 * g + 1) ^ s1));
  const uint32_t fb0 = (uint32_t)(kHalfBytes + (128 * wm + l32) * kBK + 16 * ((2 * g) ^ s1));
  const uint32_t fb1 = (uint32_t)(kHalfBytes + (128 * wm + l32) * kBK + 16 * ((2 * g + 1) ^ s1));
  auto read_frags = [&](int buf, i32x8 (&fa)[4], i32x8 (&fb)[4]) {
    const uint8_t* sb = lds + buf * kStageBytes;
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
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  auto mfma_half = [&](const i32x8 (&fa)[4], const i32x8 (&fb)[4], int half) {
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 2 * half + jj;
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa[i], fb[j], acc[i][j], 0, 0,
                                                                    0, kOneE8m0, 0, kOneE8m0);
      }
  };

  // Every stage issues the same 8 copies per wave, so each wait is one
  // constant vmcnt and the loop body is a single basic block: the copies
  // of stages past the end (index clamped to the last stage) land in
  // buffers that are never read again.
  const int S = a.K / kBK;
#pragma unroll
  for (int st = 0; st < kStages; ++st) copy_stage(min(st, S - 1), st);
  wait_vm24();  // stage 0 landed (this wave's part); stages 1..3 in flight
  barrier_keep_loads();

  i32x8 fa_c[4], fb_c[4], fa_n[4], fb_n[4];
  read_frags(0, fa_c, fb_c);

  // stage s (with a successor): first half of the MFMAs; the wait for stage
  // s+1 and the barrier that releases stage s's buffer; its refill with
  // stage s+4; the fragments of stage s+1; second half
  for (int s = 0; s + 1 < S; ++s) {
    mfma_half(fa_c, fb_c, 0);
    wait_vm16();  // stage s+1 landed; s+2 and s+3 may still be in flight
    wait_lgkm0();
    barrier_keep_loads();  // every wave has stage s+1 and is done reading stage s
    copy_stage(min(s + kStages, S - 1), s & (kStages - 1));
    read_frags((s + 1) & (kStages - 1), fa_n, fb_n);
    mfma_half(fa_c, fb_c, 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      fa_c[i] = fa_n[i];
      fb_c[i] = fb_n[i];
    }
  }
  mfma_half(fa_c, fb_c, 0);
  mfma_half(fa_c, fb_c, 1);
  wait_vm0();  // the clamped copies of the last stages

  // Epilogue through LDS, so that the stores are whole 256-byte row segments.
  // acc[i][j][4q + u] is output channel 128 wn + 32 i + 8 q + 4 g + u of
  // token 128 wm + 32 j + l32 (tile-local).  Each wave stages its 128 x 128
  // bf16 block in its own 32 KB of LDS (rows of 256 bytes, 16-byte chunk c of
  // row r at slot c ^ (r & 15)), then stores 4 rows x 256 bytes per
  // instruction.  The stage buffers are reused: every wave must be done with
  // its last fragment reads and every copy must have landed first.
  wait_lgkm0();
  barrier_keep_loads();
  uint8_t* stg = lds + wave * (kBM / 2) * 256;
  float sxv[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int m = m0 + 128 * wm + 32 * j + l32;
    sxv[j] = m < a.M ? a.sx[m] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int n = n0 + 128 * wn + 32 * i + 8 * q + 4 * g;
      f32x4 swv = {0.f, 0.f, 0.f, 0.f}, bv = {0.f, 0.f, 0.f, 0.f};
      if (n < a.N) {
        swv = *reinterpret_cast<const f32x4*>(a.sw + n);
        if (a.bias) bv = *reinterpret_cast<const f32x4*>(a.bias + n);
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int r = 32 * j + l32;
        float v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = fmaf(acc[i][j][4 * q + u] * sxv[j], swv[u], bv[u]);
        u32x2 o;
        o[0] = pack_bf16x2(v[0], v[1]);
        o[1] = pack_bf16x2(v[2], v[3]);
        *reinterpret_cast<u32x2*>(stg + r * 256 + (((4 * i + q) ^ (r & 15)) << 4) + 8 * g) = o;
      }
    }
  }
  wait_lgkm0();  // the wave reads back only what it wrote itself
  const int c = lane & 15;
  const int n = n0 + 128 * wn + 8 * c;
#pragma unroll 4
  for (int p = 0; p < 32; ++p) {
    const int r = 4 * p + (lane >> 4);
    const u32x4 v = *reinterpret_cast<const u32x4*>(stg + r * 256 + ((c ^ (r & 15)) << 4));
    const int m = m0 + 128 * wm + r;
    if (m < a.M && n < a.N) st16(a.y + (int64_t)m * a.ldy + n, v);
  }
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
  const int T = a.tiles_m * a.tiles_n;
  linear_w8a8_kernel<<<dim3((unsigned)T), 256, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace sa

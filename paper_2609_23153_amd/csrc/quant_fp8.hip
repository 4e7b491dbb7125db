// FP8 E4M3 (OCP e4m3fn) quantisation of a bf16 attention operand with one
// power-of-two scale per block of tokens, in one pass over memory (the paper
// fuses its per-token activation quantisation into one kernel for the same
// reason, §4.3).
//
// One workgroup per (batch, head, block): the block (<= 128 tokens x 128
// channels of bf16) is held in registers, its absolute maximum is reduced
// with integer compares on the bf16 magnitude bits, the scale exponent is
// chosen so that amax <= 448 * 2^e, and every value is rounded to e4m3 with
// round-to-nearest-even in integer arithmetic.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kQThreads = 256;

// Smallest e with amax <= 448 * 2^e, clamped to >= -126 so that 2^e is a
// normal fp32 (and a valid E8M0 scale code); 0 for an all-zero block.
__device__ __forceinline__ int scale_exponent(float amax) {
  if (amax == 0.f) return 0;
  int ex;
  const float fr = frexpf(amax, &ex);  // amax = fr * 2^ex, fr in [0.5, 1)
  const int e = ex - 9 + (fr > 0.875f ? 1 : 0);
  return e < -126 ? -126 : e;
}

template <int ROWS_PER_THREAD>
__global__ __launch_bounds__(kQThreads) void quant_fp8_kernel(const uint16_t* __restrict__ x,
                                                              Strides xs, int H, int N, int block,
                                                              int nb, uint8_t* __restrict__ x8,
                                                              float* __restrict__ scale) {
  const int bh = blockIdx.y, i = blockIdx.x;
  const int b = bh / H, h = bh - b * H;
  const int t0 = i * block;
  const int n_i = min(block, N - t0);
  const int chunk = threadIdx.x & 15, r0 = threadIdx.x >> 4;
  const uint16_t* src = x + b * xs.b + h * xs.h;

  u32x4 v[ROWS_PER_THREAD];
  uint32_t amax = 0;  // bf16 magnitude bits; integer order = value order
#pragma unroll
  for (int m = 0; m < ROWS_PER_THREAD; ++m) {
    const int r = r0 + 16 * m;
    if (r < n_i) {
      v[m] = ld16(src + (int64_t)(t0 + r) * xs.n + chunk * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        amax = max(amax, v[m][e] & 0x7fffu);
        amax = max(amax, (v[m][e] >> 16) & 0x7fffu);
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, o, kWave));
  __shared__ uint32_t red[kQThreads / kWave];
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = amax;
  __syncthreads();
  amax = max(max(red[0], red[1]), max(red[2], red[3]));

  const int e = scale_exponent(__uint_as_float(amax << 16));
  const float inv = __uint_as_float((uint32_t)(127 - e) << 23);  // 2^-e, normal for e in [-126, 127)
  if (threadIdx.x == 0) scale[(int64_t)bh * nb + i] = __uint_as_float((uint32_t)(e + 127) << 23);

  uint8_t* dst = x8 + ((int64_t)bh * N + t0) * kHeadDim + chunk * 8;
#pragma unroll
  for (int m = 0; m < ROWS_PER_THREAD; ++m) {
    const int r = r0 + 16 * m;
    if (r < n_i) {
      u32x2 out;
#pragma unroll
      for (int hw = 0; hw < 2; ++hw) {
        const uint32_t w0 = v[m][2 * hw], w1 = v[m][2 * hw + 1];
        out[hw] = e4m3_rne(bf16_lo(w0) * inv) | (e4m3_rne(bf16_hi(w0) * inv) << 8) |
                  (e4m3_rne(bf16_lo(w1) * inv) << 16) | (e4m3_rne(bf16_hi(w1) * inv) << 24);
      }
      *reinterpret_cast<u32x2*>(dst + (int64_t)r * kHeadDim) = out;
    }
  }
}

// The same codes and scales, written in the fp8 forward's operand order: per
// (batch, head) ceil(N / 64) tiles of 64 keys x 128 channels, 8 KB each, laid
// out so that every 16-byte piece a lane loads for one matrix-core operand is
// contiguous with its neighbours' (the forward then reads 1 KB per load
// instruction and needs no LDS).  Byte (c, e) of 16-byte chunk
//   K: c = ((2 rt + ks) 2 + hf) 64 + l32 + 32 g  ->  key 32 rt + l32,
//      channel 64 ks + 32 g + 16 hf + e
//   V: c = (2 dt + hf) 64 + l32 + 32 g  ->  channel 32 dt + l32,
//      key 32 hf + 8 (e / 4) + 4 g + e % 4
// (the V order matches the order in which the forward packs probabilities).
// Keys past N are code 0.  The block's codes are staged in LDS row-major.
template <int ROWS_PER_THREAD>
__global__ __launch_bounds__(kQThreads) void quant_fp8_tiles_kernel(
    const uint16_t* __restrict__ x, Strides xs, int H, int N, int block, int nb, bool is_v,
    uint8_t* __restrict__ x8, float* __restrict__ scale) {
  constexpr int kRows = ROWS_PER_THREAD * 16;  // tokens of a block
  __shared__ __attribute__((aligned(16))) uint8_t codes[kRows * kHeadDim];
  const int bh = blockIdx.y, i = blockIdx.x;
  const int b = bh / H, h = bh - b * H;
  const int t0 = i * block;
  const int n_i = min(block, N - t0);
  const int chunk = threadIdx.x & 15, r0 = threadIdx.x >> 4;
  const uint16_t* src = x + b * xs.b + h * xs.h;

  u32x4 v[ROWS_PER_THREAD];
  uint32_t amax = 0;
#pragma unroll
  for (int m = 0; m < ROWS_PER_THREAD; ++m) {
    const int r = r0 + 16 * m;
    v[m] = (u32x4){0u, 0u, 0u, 0u};
    if (r < n_i) {
      v[m] = ld16(src + (int64_t)(t0 + r) * xs.n + chunk * 8);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        amax = max(amax, v[m][e] & 0x7fffu);
        amax = max(amax, (v[m][e] >> 16) & 0x7fffu);
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) amax = max(amax, (uint32_t)__shfl_xor((int)amax, o, kWave));
  __shared__ uint32_t red[kQThreads / kWave];
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = amax;
  __syncthreads();
  amax = max(max(red[0], red[1]), max(red[2], red[3]));
  const int e = scale_exponent(__uint_as_float(amax << 16));
  const float inv = __uint_as_float((uint32_t)(127 - e) << 23);
  if (threadIdx.x == 0) scale[(int64_t)bh * nb + i] = __uint_as_float((uint32_t)(e + 127) << 23);
  // codes row-major in LDS (rows past the end hold zeros: e4m3(0) = 0)
#pragma unroll
  for (int m = 0; m < ROWS_PER_THREAD; ++m) {
    const int r = r0 + 16 * m;
    u32x2 out;
#pragma unroll
    for (int hw = 0; hw < 2; ++hw) {
      const uint32_t w0 = v[m][2 * hw], w1 = v[m][2 * hw + 1];
      out[hw] = e4m3_rne(bf16_lo(w0) * inv) | (e4m3_rne(bf16_hi(w0) * inv) << 8) |
                (e4m3_rne(bf16_lo(w1) * inv) << 16) | (e4m3_rne(bf16_hi(w1) * inv) << 24);
    }
    *reinterpret_cast<u32x2*>(codes + r * kHeadDim + chunk * 8) = out;
  }
  __syncthreads();
  // 512 chunks of 16 bytes per 64-key tile; tiles wholly past N are skipped
  const int ntiles = (N + kTile - 1) / kTile;
  for (int tt = 0; tt < kRows / kTile; ++tt) {
    const int t = t0 / kTile + tt;
    if (tt * kTile >= block || t >= ntiles) break;
    uint8_t* dst = x8 + ((int64_t)bh * ntiles + t) * (kTile * kHeadDim);
    const uint8_t* tile = codes + tt * kTile * kHeadDim;
    for (int c = threadIdx.x; c < kTile * kHeadDim / 16; c += kQThreads) {
      const int lane = c & 63, l32 = lane & 31, g = lane >> 5;
      u32x4 w;
      if (!is_v) {
        const int hf = (c >> 6) & 1, ks = (c >> 7) & 1, rt = c >> 8;
        w = *reinterpret_cast<const u32x4*>(tile + (32 * rt + l32) * kHeadDim + 64 * ks + 32 * g +
                                            16 * hf);
      } else {
        const int hf = (c >> 6) & 1, dt = c >> 7;
        const uint8_t* col = tile + 32 * dt + l32;
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const int k0 = 32 * hf + 8 * q4 + 4 * g;
          w[q4] = (uint32_t)col[k0 * kHeadDim] | ((uint32_t)col[(k0 + 1) * kHeadDim] << 8) |
                  ((uint32_t)col[(k0 + 2) * kHeadDim] << 16) |
                  ((uint32_t)col[(k0 + 3) * kHeadDim] << 24);
        }
      }
      st16(dst + c * 16, w);
    }
  }
}

}  // namespace

hipError_t launch_quant_fp8_tiles(const Shape& s, const void* x, Strides xs, bool is_v,
                                  uint8_t* x8, float* scale, hipStream_t stream) {
  const dim3 grid(s.nb, s.B * s.H);
  const uint16_t* xp = static_cast<const uint16_t*>(x);
  if (s.block == 64)
    quant_fp8_tiles_kernel<4><<<grid, kQThreads, 0, stream>>>(xp, xs, s.H, s.N, s.block, s.nb,
                                                              is_v, x8, scale);
  else
    quant_fp8_tiles_kernel<8><<<grid, kQThreads, 0, stream>>>(xp, xs, s.H, s.N, s.block, s.nb,
                                                              is_v, x8, scale);
  return hipGetLastError();
}

hipError_t launch_quant_fp8(const Shape& s, const void* x, Strides xs, uint8_t* x8, float* scale,
                            hipStream_t stream) {
  const dim3 grid(s.nb, s.B * s.H);
  const uint16_t* xp = static_cast<const uint16_t*>(x);
  if (s.block == 64)
    quant_fp8_kernel<4><<<grid, kQThreads, 0, stream>>>(xp, xs, s.H, s.N, s.block, s.nb, x8, scale);
  else
    quant_fp8_kernel<8><<<grid, kQThreads, 0, stream>>>(xp, xs, s.H, s.N, s.block, s.nb, x8, scale);
  return hipGetLastError();
}

}  // namespace sa

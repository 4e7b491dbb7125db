// Block selection M_phi on gfx950 (paper §2 Eq. comp-sparse; selection kept
// in BF16 inputs per §4.3): mean-pooled block scores and per-query-block
// top-k with ties to the lower block index.
//
// Three launches:
//   pool   : Q and K streamed once from HBM; per block, the fp64 sum of the
//            bf16 token vectors (exact for bf16 inputs whose exponents span
//            fewer than ~38 binades, so it does not depend on summation order)
//   score  : per (batch, head) an fp64 GEMM qhat . khat^T scaled by
//            1 / (n_i n_j)  -> scores in the workspace
//   topk   : one wavefront per query block; a bitwise radix search over
//            order-preserving 64-bit keys finds the k-th largest score, then
//            ballots emit the kept block indices in ascending order.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kPoolThreads = 256;

// One workgroup pools one block of Q (blockIdx.z == 0) or K (== 1).
__global__ __launch_bounds__(kPoolThreads) void pool_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, Strides qs, Strides ks,
    int H, int N, int block, int nb, double* __restrict__ qhat, double* __restrict__ khat) {
  const bool is_k = blockIdx.z != 0;
  const uint16_t* x = is_k ? k : q;
  const Strides st = is_k ? ks : qs;
  double* out = is_k ? khat : qhat;
  const int bh = blockIdx.y;
  const int b = bh / H, h = bh - b * H;
  const int i = blockIdx.x;
  const int t0 = i * block;
  const int n_i = min(block, N - t0);
  const uint16_t* base = x + b * st.b + h * st.h + (int64_t)t0 * st.n;

  const int col8 = threadIdx.x & 15;  // 8 channels = 16 bytes
  const int r0 = threadIdx.x >> 4;    // 16 row groups
  double acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = 0.0;
  for (int r = r0; r < n_i; r += 16) {
    const u32x4 w = ld16(base + (int64_t)r * st.n + col8 * 8);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += (double)bf16_lo(w[e]);
      acc[2 * e + 1] += (double)bf16_hi(w[e]);
    }
  }
  __shared__ double red[16][kHeadDim + 1];
#pragma unroll
  for (int c = 0; c < 8; ++c) red[r0][col8 * 8 + c] = acc[c];
  __syncthreads();
  if (threadIdx.x < kHeadDim) {
    double s = 0.0;
#pragma unroll
    for (int r = 0; r < 16; ++r) s += red[r][threadIdx.x];
    out[((int64_t)bh * nb + i) * kHeadDim + threadIdx.x] = s;
  }
}

// fp64 score GEMM: one 64x64 tile of S = qhat khat^T / (n_i n_j) per workgroup.
constexpr int kSTile = 64;
constexpr int kSK = 32;  // depth staged per step
__global__ __launch_bounds__(256) void score_kernel(const double* __restrict__ qhat,
                                                   const double* __restrict__ khat, int N,
                                                   int block, int nb,
                                                   double* __restrict__ scores) {
  const int bh = blockIdx.z;
  const int i0 = blockIdx.y * kSTile, j0 = blockIdx.x * kSTile;
  const double* qb = qhat + (int64_t)bh * nb * kHeadDim;
  const double* kb = khat + (int64_t)bh * nb * kHeadDim;
  __shared__ double As[kSK][kSTile + 1];
  __shared__ double Bs[kSK][kSTile + 1];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  double acc[4][4];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < 4; ++c) acc[r][c] = 0.0;

  const int lr = threadIdx.x >> 2;       // tile row loaded by this thread
  const int lk = (threadIdx.x & 3) * 8;  // 8 consecutive depth values
  for (int k0 = 0; k0 < kHeadDim; k0 += kSK) {
    const bool qa = i0 + lr < nb, ka = j0 + lr < nb;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      As[lk + e][lr] = qa ? qb[(int64_t)(i0 + lr) * kHeadDim + k0 + lk + e] : 0.0;
      Bs[lk + e][lr] = ka ? kb[(int64_t)(j0 + lr) * kHeadDim + k0 + lk + e] : 0.0;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < kSK; ++kk) {
      double a[4], bv[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) a[r] = As[kk][ty + 16 * r];
#pragma unroll
      for (int c = 0; c < 4; ++c) bv[c] = Bs[kk][tx + 16 * c];
#pragma unroll
      for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[r][c] = fma(a[r], bv[c], acc[r][c]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = i0 + ty + 16 * r;
    if (i >= nb) continue;
    const int n_i = min(block, N - i * block);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int j = j0 + tx + 16 * c;
      if (j >= nb) continue;
      const int n_j = min(block, N - j * block);
      scores[((int64_t)bh * nb + i) * nb + j] = acc[r][c] / (double)(n_i * n_j);
    }
  }
}

// Order-preserving map of a double to uint64 (larger score -> larger key);
// -0 and +0 map to the same key.  0 is below every finite score (padding).
__device__ __forceinline__ uint64_t order_key(double s) {
  if (s == 0.0) s = 0.0;
  const uint64_t u = (uint64_t)__double_as_longlong(s);
  return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint64_t y = __shfl_xor(x, o, kWave);
    x = y > x ? y : x;
  }
  return x;
}
__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint64_t y = __shfl_xor(x, o, kWave);
    x = y < x ? y : x;
  }
  return x;
}

// k-th largest key (with multiplicity) of the wave's keys: the largest T with
// count(key >= T) >= k.  Stops early once some prefix selects exactly k keys
// (then every key >= T is kept, ties included).
template <int KPL>
__device__ __forceinline__ uint64_t kth_largest(const uint64_t (&key)[KPL], const bool (&valid)[KPL],
                                                int k) {
  uint64_t mx = 0, mn = ~0ull;
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    if (valid[t]) {
      mx = key[t] > mx ? key[t] : mx;
      mn = key[t] < mn ? key[t] : mn;
    }
  }
  mx = wave_max_u64(mx);
  mn = wave_min_u64(mn);
  if (mx == mn) return mx;
  const int top = 63 - __clzll(mx ^ mn);
  uint64_t prefix = mx & ~((2ull << top) - 1ull);  // bits above `top` are common
  for (int bit = top; bit >= 0; --bit) {
    const uint64_t cand = prefix | (1ull << bit);
    int c = 0;
#pragma unroll
    for (int t = 0; t < KPL; ++t) c += (valid[t] && key[t] >= cand) ? 1 : 0;
    c = wave_sum(c);
    if (c >= k) {
      prefix = cand;
      if (c == k) break;
    }
  }
  return prefix;
}

template <int KPL>
__global__ __launch_bounds__(256) void topk_row_kernel(const double* __restrict__ scores,
                                                       int nb, int rows, int k, int kmax,
                                                       int32_t* __restrict__ idx,
                                                       int32_t* __restrict__ cnt) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;  // uniform per wave
  const double* s = scores + (int64_t)row * nb;
  uint64_t key[KPL];
  bool valid[KPL];
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    const int j = lane + kWave * t;
    valid[t] = j < nb;
    key[t] = valid[t] ? order_key(s[j]) : 0ull;
  }
  const uint64_t thr = kth_largest<KPL>(key, valid, k);
  int gt = 0;
#pragma unroll
  for (int t = 0; t < KPL; ++t) gt += (valid[t] && key[t] > thr) ? 1 : 0;
  const int need_eq = k - wave_sum(gt);  // ties at the threshold, lowest index first

  const uint64_t below = lanes_below_mask();
  int32_t* out = idx + (int64_t)row * kmax;
  int taken = 0, eq_seen = 0;
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    const int j = lane + kWave * t;
    const bool eq = valid[t] && key[t] == thr;
    const uint64_t eq_mask = __ballot(eq);
    const int eq_rank = eq_seen + __popcll(eq_mask & below);
    const bool sel = (valid[t] && key[t] > thr) || (eq && eq_rank < need_eq);
    const uint64_t sel_mask = __ballot(sel);
    if (sel) out[taken + __popcll(sel_mask & below)] = j;
    taken += __popcll(sel_mask);
    eq_seen += __popcll(eq_mask);
  }
  for (int p = k + lane; p < kmax; p += kWave) out[p] = -1;
  if (lane == 0) cnt[row] = k;
}

template <int KPL>
hipError_t launch_topk(const double* scores, int nb, int rows, int k, int kmax, int32_t* idx,
                       int32_t* cnt, hipStream_t stream) {
  topk_row_kernel<KPL><<<(rows + 3) / 4, 256, 0, stream>>>(scores, nb, rows, k, kmax, idx, cnt);
  return hipGetLastError();
}

}  // namespace

size_t select_workspace_bytes(const Shape& s) {
  const size_t bh = (size_t)s.B * s.H;
  return bh * s.nb * kHeadDim * sizeof(double) * 2 + bh * s.nb * s.nb * sizeof(double);
}

static hipError_t launch_pool_score(const Shape& s, const void* q, Strides qs, const void* k,
                                    Strides ks, void* ws, double** scores_out,
                                    hipStream_t stream) {
  const size_t bh = (size_t)s.B * s.H;
  double* qhat = static_cast<double*>(ws);
  double* khat = qhat + bh * s.nb * kHeadDim;
  double* scores = khat + bh * s.nb * kHeadDim;
  pool_kernel<<<dim3(s.nb, bh, 2), kPoolThreads, 0, stream>>>(
      static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), qs, ks, s.H, s.N,
      s.block, s.nb, qhat, khat);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int tiles = (s.nb + kSTile - 1) / kSTile;
  score_kernel<<<dim3(tiles, tiles, bh), 256, 0, stream>>>(qhat, khat, s.N, s.block, s.nb,
                                                           scores);
  *scores_out = scores;
  return hipGetLastError();
}

hipError_t launch_select_row(const Shape& s, const void* q, Strides qs, const void* k,
                             Strides ks, int topk, int kmax, int32_t* idx, int32_t* cnt,
                             void* ws, hipStream_t stream) {
  double* scores = nullptr;
  hipError_t e = launch_pool_score(s, q, qs, k, ks, ws, &scores, stream);
  if (e != hipSuccess) return e;
  const int rows = s.B * s.H * s.nb;
  const int kpl = (s.nb + kWave - 1) / kWave;
  if (kpl <= 1) return launch_topk<1>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 2) return launch_topk<2>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 4) return launch_topk<4>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 8) return launch_topk<8>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 16) return launch_topk<16>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 24) return launch_topk<24>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 32) return launch_topk<32>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  return launch_topk<64>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
}

hipError_t launch_select_head(const Shape&, const void*, Strides, const void*, Strides,
                              int64_t, int, int32_t*, int32_t*, void*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace sa

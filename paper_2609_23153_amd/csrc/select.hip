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
//   topk   : one wavefront per query block; a bitwise search over
//            order-preserving 64-bit keys (high word first, then the low word
//            of the keys tied there) finds the k-th largest score, then
//            ballots emit the kept block indices in ascending order.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kPoolThreads = 256;
constexpr int kMaxBlock = 128;  // largest supported block size

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
  // block <= 128: at most 8 rows per thread, all loads issued before the sums
  u32x4 w[kMaxBlock / 16];
#pragma unroll
  for (int m = 0; m < kMaxBlock / 16; ++m) {
    const int r = r0 + 16 * m;
    w[m] = r < n_i ? ld16(base + (int64_t)r * st.n + col8 * 8) : (u32x4){0u, 0u, 0u, 0u};
  }
#pragma unroll
  for (int m = 0; m < kMaxBlock / 16; ++m)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] += (double)bf16_lo(w[m][e]);
      acc[2 * e + 1] += (double)bf16_hi(w[m][e]);
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

// fp64 score GEMM on the matrix cores: one 64x64 tile of
// S = qhat khat^T / (n_i n_j) per workgroup of 4 waves, each wave a 32x32
// quarter as 2x2 v_mfma_f64_16x16x4f64 tiles.  qhat and khat are staged
// through LDS in 32-deep slices, [row][k] with a row stride of 34 doubles
// (conflict-free both for the 16-byte row-contiguous stores and for the
// operand reads, 16 rows x 2 depths per half-wave).  The next slice is
// fetched into registers (16-byte loads, all in flight together) while the
// current one is multiplied.  The results are fp64 roundings of the dot
// products in an order that differs from the oracle's only in the last bits.
constexpr int kSTile = 64;
constexpr int kSDepth = 32;
constexpr int kSStride = 34;
constexpr int kSChunks = kSTile * kSDepth / 2 / 256;  // 16-byte chunks per thread per operand
typedef __attribute__((__vector_size__(4 * sizeof(double)))) double f64x4;
typedef __attribute__((__vector_size__(2 * sizeof(double)))) double f64x2;

__global__ __launch_bounds__(256) void score_kernel(const double* __restrict__ qhat,
                                                   const double* __restrict__ khat, int N,
                                                   int block, int nb,
                                                   double* __restrict__ scores) {
  const int bh = blockIdx.z;
  const int i0 = blockIdx.y * kSTile, j0 = blockIdx.x * kSTile;
  const double* qb = qhat + (int64_t)bh * nb * kHeadDim;
  const double* kb = khat + (int64_t)bh * nb * kHeadDim;
  __shared__ __attribute__((aligned(16))) double As[kSTile * kSStride];
  __shared__ __attribute__((aligned(16))) double Bs[kSTile * kSStride];
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const int wr = (w >> 1) * 32, wc = (w & 1) * 32;  // this wave's 32x32 quarter
  // 16x16x4 f64 operands: A lane l holds A[l%16][l/16], B lane l holds B[l/16][l%16];
  // D lane l holds D[l/16 + 4r][l%16], r = 0..3.
  const int li = l & 15, lk = l >> 4;
  f64x4 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c) acc[a][c] = (f64x4){0.0, 0.0, 0.0, 0.0};

  // thread t moves chunk e = t + 256m: tile row e / 16, depth 2 * (e % 16)
  f64x2 ra[kSChunks], rb[kSChunks];
  auto fetch = [&](int k0) {
#pragma unroll
    for (int m = 0; m < kSChunks; ++m) {
      const int e = threadIdx.x + 256 * m;
      const int r = e >> 4, c = 2 * (e & 15);
      const f64x2 z = {0.0, 0.0};
      ra[m] = i0 + r < nb ? *reinterpret_cast<const f64x2*>(qb + (int64_t)(i0 + r) * kHeadDim + k0 + c) : z;
      rb[m] = j0 + r < nb ? *reinterpret_cast<const f64x2*>(kb + (int64_t)(j0 + r) * kHeadDim + k0 + c) : z;
    }
  };
  auto stage = [&]() {
#pragma unroll
    for (int m = 0; m < kSChunks; ++m) {
      const int e = threadIdx.x + 256 * m;
      const int r = e >> 4, c = 2 * (e & 15);
      *reinterpret_cast<f64x2*>(&As[r * kSStride + c]) = ra[m];
      *reinterpret_cast<f64x2*>(&Bs[r * kSStride + c]) = rb[m];
    }
  };
  fetch(0);
  stage();
  __syncthreads();
  for (int k0 = 0; k0 < kHeadDim; k0 += kSDepth) {
    if (k0 + kSDepth < kHeadDim) fetch(k0 + kSDepth);
#pragma unroll
    for (int kk = 0; kk < kSDepth; kk += 4) {
      const double a0 = As[(wr + li) * kSStride + kk + lk];
      const double a1 = As[(wr + 16 + li) * kSStride + kk + lk];
      const double b0 = Bs[(wc + li) * kSStride + kk + lk];
      const double b1 = Bs[(wc + 16 + li) * kSStride + kk + lk];
      acc[0][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f64_16x16x4f64(a1, b1, acc[1][1], 0, 0, 0);
    }
    if (k0 + kSDepth < kHeadDim) {
      __syncthreads();
      stage();
      __syncthreads();
    }
  }
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int c = 0; c < 2; ++c)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = i0 + wr + 16 * a + lk + 4 * r;
        const int j = j0 + wc + 16 * c + li;
        if (i < nb && j < nb) {
          const int n_i = min(block, N - i * block), n_j = min(block, N - j * block);
          scores[((int64_t)bh * nb + i) * nb + j] = acc[a][c][r] / (double)(n_i * n_j);
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

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = max(x, (uint32_t)__shfl_xor((int)x, o, kWave));
  return x;
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = min(x, (uint32_t)__shfl_xor((int)x, o, kWave));
  return x;
}

// Largest 32-bit T with count(member && v >= T) >= k over the wave (the k-th
// largest member value, with multiplicity), by a bitwise search from the
// highest bit in which the members differ.  Stops early once a prefix
// selects exactly k values; *exact is then set (every member >= T is kept).
// Requires 1 <= k <= count(member).
template <int KPL>
__device__ __forceinline__ uint32_t kth_largest32(const uint32_t (&v)[KPL], const bool (&member)[KPL],
                                                  int k, bool* exact) {
  uint32_t mx = 0, mn = ~0u;
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    if (member[t]) {
      mx = max(mx, v[t]);
      mn = min(mn, v[t]);
    }
  }
  mx = wave_max_u32(mx);
  mn = wave_min_u32(mn);
  *exact = false;
  if (mx == mn) return mx;
  const int top = 31 - __clz(mx ^ mn);
  uint32_t prefix = top == 31 ? 0u : mx & ~((2u << top) - 1u);  // bits above `top` are common
  for (int bit = top; bit >= 0; --bit) {
    const uint32_t cand = prefix | (1u << bit);
    // count over the wave with ballots: scalar popcounts, no cross-lane shuffles
    int c = 0;
#pragma unroll
    for (int t = 0; t < KPL; ++t) c += __popcll(__ballot(member[t] && v[t] >= cand));
    if (c >= k) {
      prefix = cand;
      if (c == k) {
        *exact = true;
        break;
      }
    }
  }
  return prefix;
}

// One wavefront per query block: the k largest of the row's order keys
// (64-bit), ties to the lower block index, emitted in ascending index order.
// The k-th largest key is found on its high 32 bits first; only the keys that
// tie with it there take part in the search over the low 32 bits.
template <int KPL>
__global__ __launch_bounds__(256) void topk_row_kernel(const double* __restrict__ scores,
                                                       int nb, int rows, int k, int kmax,
                                                       int32_t* __restrict__ idx,
                                                       int32_t* __restrict__ cnt) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;  // uniform per wave
  const double* s = scores + (int64_t)row * nb;
  uint32_t hi[KPL], lo[KPL];
  bool valid[KPL];
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    const int j = lane + kWave * t;
    valid[t] = j < nb;
    const uint64_t key = valid[t] ? order_key(s[j]) : 0ull;
    hi[t] = (uint32_t)(key >> 32);
    lo[t] = (uint32_t)key;
  }
  bool exact;
  const uint32_t thi = kth_largest32<KPL>(hi, valid, k, &exact);
  // selection: hi > thi, or hi == thi and (lo > tlo, or lo == tlo and among
  // the first need_eq such keys in index order)
  uint32_t tlo = 0;
  int need_eq = 0;
  if (!exact) {
    int gt = 0;
#pragma unroll
    for (int t = 0; t < KPL; ++t) gt += __popcll(__ballot(valid[t] && hi[t] > thi));
    bool grp[KPL];
#pragma unroll
    for (int t = 0; t < KPL; ++t) grp[t] = valid[t] && hi[t] == thi;
    bool ex2;
    tlo = kth_largest32<KPL>(lo, grp, k - gt, &ex2);
    int gt2 = 0;
#pragma unroll
    for (int t = 0; t < KPL; ++t) gt2 += __popcll(__ballot(grp[t] && lo[t] > tlo));
    need_eq = k - gt - gt2;
  }

  const uint64_t below = lanes_below_mask();
  int32_t* out = idx + (int64_t)row * kmax;
  int taken = 0, eq_seen = 0;
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    const int j = lane + kWave * t;
    bool sel;
    if (exact) {
      sel = valid[t] && hi[t] >= thi;
    } else {
      const bool eq = valid[t] && hi[t] == thi && lo[t] == tlo;
      const uint64_t eq_mask = __ballot(eq);
      const int eq_rank = eq_seen + __popcll(eq_mask & below);
      sel = (valid[t] && (hi[t] > thi || (hi[t] == thi && lo[t] > tlo))) ||
            (eq && eq_rank < need_eq);
      eq_seen += __popcll(eq_mask);
    }
    const uint64_t sel_mask = __ballot(sel);
    if (sel) out[taken + __popcll(sel_mask & below)] = j;
    taken += __popcll(sel_mask);
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
  if (kpl <= 12) return launch_topk<12>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 16) return launch_topk<16>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 20) return launch_topk<20>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 24) return launch_topk<24>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  if (kpl <= 32) return launch_topk<32>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
  return launch_topk<64>(scores, s.nb, rows, topk, kmax, idx, cnt, stream);
}

hipError_t launch_select_head(const Shape&, const void*, Strides, const void*, Strides,
                              int64_t, int, int32_t*, int32_t*, void*, hipStream_t) {
  return hipErrorNotSupported;
}

}  // namespace sa

// Block selection M_phi on gfx950 (paper §2 Eq. comp-sparse; selection kept
// in BF16 inputs per §4.3): mean-pooled block scores and per-query-block
// top-k with ties to the lower block index, or the ragged whole-head variant.
//
// Launches:
//   pool   : Q and K streamed once from HBM; per block, the fp64 sum of the
//            bf16 token vectors (exact for bf16 inputs whose exponents span
//            fewer than ~38 binades, so it does not depend on summation order)
//   row mode, nb <= kFStrideBig (the scores never reach HBM): pool of K only,
//   score_topk : per 32 query blocks, their pooling (same arithmetic as the
//            pool launch), then approximate scores of every key block
//            on the bf16 matrix cores from a two-term bf16 split of the
//            pooled sums, kept in LDS; per query block the k-th largest
//            approximation and a rigorous error bound split the key blocks
//            into certainly kept, certainly dropped and a band between; only
//            the band is rescored in fp64 (see the comment above
//            score_topk_kernel)
//   otherwise:
//   score  : per (batch, head) an fp64 GEMM qhat . khat^T scaled by
//            1 / (n_i n_j)  -> scores in the workspace
//   topk   : one wavefront per query block; a bitwise search over
//            order-preserving 64-bit keys (high word first, then the low word
//            of the keys tied there) finds the k-th largest score, then
//            ballots emit the kept block indices in ascending order.
//   whole-head mode: row bests, an 8-pass radix select of the global
//            threshold key per head, per-row counts and a scan, then the row
//            top-k with a per-row k (see the comment above head_init_kernel).
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

typedef __attribute__((__vector_size__(4 * sizeof(double)))) double f64x4;
typedef __attribute__((__vector_size__(2 * sizeof(double)))) double f64x2;

// x of the lane N places lower within its row of 16 lanes (cyclically), by
// DPP: no LDS round trip.  `idle` is returned for a disabled source lane.
template <int N>
__device__ __forceinline__ uint32_t row_ror(uint32_t x, uint32_t idle) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)idle, (int)x, 0x120 + N, 0xF, 0xF, false);
}
// Number of set bits of m below this lane (v_mbcnt).
__device__ __forceinline__ int rank_below(uint64_t m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
// Whole-wave max / min, the result in every lane (a wave-uniform value): a
// butterfly over the 16 lanes of a row, then over rows through
// v_permlane16_swap / 32_swap.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  x = max(x, row_ror<8>(x, 0u));
  x = max(x, row_ror<4>(x, 0u));
  x = max(x, row_ror<2>(x, 0u));
  x = max(x, row_ror<1>(x, 0u));
  const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = max(a[0], a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return __builtin_amdgcn_readfirstlane(max(b[0], b[1]));  // the same in every lane
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
  x = min(x, row_ror<8>(x, ~0u));
  x = min(x, row_ror<4>(x, ~0u));
  x = min(x, row_ror<2>(x, ~0u));
  x = min(x, row_ror<1>(x, ~0u));
  const auto a = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = min(a[0], a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return __builtin_amdgcn_readfirstlane(min(b[0], b[1]));
}
// fp64 x of lane l plus x of lane l ^ 16 (XOR16) or l ^ 32.
template <bool XOR16>
__device__ __forceinline__ double add_swapped(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = (uint32_t)u, hi = (uint32_t)(u >> 32);
  const auto l2 = XOR16 ? __builtin_amdgcn_permlane16_swap(lo, lo, false, false)
                        : __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
  const auto h2 = XOR16 ? __builtin_amdgcn_permlane16_swap(hi, hi, false, false)
                        : __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
  const double a = __longlong_as_double((long long)(((uint64_t)h2[0] << 32) | l2[0]));
  const double b = __longlong_as_double((long long)(((uint64_t)h2[1] << 32) | l2[1]));
  return a + b;
}
template <int N>
__device__ __forceinline__ double row_ror_f64(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = row_ror<N>((uint32_t)u, 0u), hi = row_ror<N>((uint32_t)(u >> 32), 0u);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// Whole-wave fp64 sum (every lane gets a sum of all 64 values, in a
// lane-dependent but fixed order).
__device__ __forceinline__ double wave_sum_f64(double x) {
  x += row_ror_f64<8>(x);
  x += row_ror_f64<4>(x);
  x += row_ror_f64<2>(x);
  x += row_ror_f64<1>(x);
  x = add_swapped<true>(x);
  return add_swapped<false>(x);
}

// Fused row selection: query blocks per workgroup, and the 16-deep k-steps of
// the split operands (steps 0..7: high parts of channels 16 s .. 16 s + 15,
// steps 8..15: low parts of the same channels).
constexpr int kFRows = 32;
constexpr int kFSteps = 16;

// Smallest fp32 >= x (x >= 0 or NaN).
__device__ __forceinline__ float f32_round_up(double x) {
  float f = (float)x;
  if ((double)f < x) f = __uint_as_float(__float_as_uint(f) + 1u);
  return f;
}

// Outputs of the K pooling besides the fp64 sums, for the fused row
// selection (null otherwise): the sums split as hi + lo, hi = bf16(sum) and
// lo = bf16(sum - hi), in MFMA operand order
// [B*H][tile of 32 blocks][k-step][lane][8 channels] (lane = block % 32 +
// 32 * (channel / 8 % 2)), and norm[b] = |sum| / n_b rounded up to fp32.
struct PoolSplit {
  uint16_t* frag;
  float* norm;
  int ntiles;  // ceil(nb / 32)
};

// Pooled sums of the block of tokens [t0, t0 + BLOCK) ∩ [0, N) of one head
// (x: its token 0) by one wave: lane l loads 16 bytes (channels
// 8 (l % 16) .. +7) of rows l / 16, l / 16 + 4, ..., all loads in flight
// before the fp64 sums; the four row groups are then added across lanes
// (v_permlane16 / 32_swap), so every lane ends with the block's sums of its 8
// channels (exact: the order does not matter).  Rows past N load token N - 1
// (no branch around the loads, which would make the compiler wait on each)
// and count as zero.
template <int BLOCK>
__device__ __forceinline__ void pool_load(const uint16_t* __restrict__ x, int64_t stride_n,
                                          int t0, int N, u32x4 (&w)[BLOCK / 4]) {
  const int lane = threadIdx.x & (kWave - 1);
  const int c8 = lane & 15, r0 = lane >> 4;
#pragma unroll
  for (int m = 0; m < BLOCK / 4; ++m)
    w[m] = ld16(x + (int64_t)min(t0 + r0 + 4 * m, N - 1) * stride_n + c8 * 8);
  __builtin_amdgcn_sched_barrier(0);  // every load issued before the sums start
}
template <int BLOCK>
__device__ __forceinline__ void pool_reduce(const u32x4 (&w)[BLOCK / 4], int t0, int N,
                                            double (&acc)[8]) {
  const int r0 = (threadIdx.x & (kWave - 1)) >> 4;
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = 0.0;
#pragma unroll
  for (int m = 0; m < BLOCK / 4; ++m) {
    const bool in = t0 + r0 + 4 * m < N;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t v = in ? w[m][e] : 0u;
      acc[2 * e] += (double)bf16_lo(v);
      acc[2 * e + 1] += (double)bf16_hi(v);
    }
  }
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = add_swapped<false>(add_swapped<true>(acc[c]));
}
template <int BLOCK>
__device__ __forceinline__ void pool_sums(const uint16_t* __restrict__ x, int64_t stride_n,
                                          int t0, int N, double (&acc)[8]) {
  u32x4 w[BLOCK / 4];
  pool_load<BLOCK>(x, stride_n, t0, N, w);
  pool_reduce<BLOCK>(w, t0, N, acc);
}

// The split of 8 pooled sums s = hi + lo + rest, packed as bf16 (|s - hi| <=
// 2^-8 |s| after the fp32 then bf16 roundings, up to 2^-23 more; s - hi exact
// in fp64; |rest| <= 2^-16 |s| (1 + 2^-14)), and the sum of their squares.
__device__ __forceinline__ void split_hi_lo(const double (&acc)[8], u32x4& whi, u32x4& wlo,
                                            double& sq) {
  sq = 0.0;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    uint32_t hh[2], ll[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const double sv = acc[2 * e + u];
      hh[u] = f32_to_bf16_rne((float)sv);
      ll[u] = f32_to_bf16_rne((float)(sv - (double)__uint_as_float(hh[u] << 16)));
      sq = fma(sv, sv, sq);
    }
    whi[e] = hh[0] | (hh[1] << 16);
    wlo[e] = ll[0] | (ll[1] << 16);
  }
}

// |sum|^2 over the 16 lanes of a row (each row of lanes holds all 128 channels)
__device__ __forceinline__ double row_sum16(double x) {
  x += row_ror_f64<8>(x);
  x += row_ror_f64<4>(x);
  x += row_ror_f64<2>(x);
  x += row_ror_f64<1>(x);
  return x;
}

// One wave pools one block of Q (blockIdx.z + z0 == 0) or K (== 1); a
// workgroup takes 4 consecutive blocks of one (batch, head).  No LDS.
constexpr int kPoolWaves = 4;

template <int BLOCK>
__global__ __launch_bounds__(kPoolWaves * kWave) void pool_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, Strides qs, Strides ks,
    int H, int N, int nb, int z0, double* __restrict__ qhat, double* __restrict__ khat,
    PoolSplit split) {
  const bool is_k = (int)blockIdx.z + z0 != 0;
  const uint16_t* x = is_k ? k : q;
  const Strides st = is_k ? ks : qs;
  double* out = is_k ? khat : qhat;
  const int bh = blockIdx.y;
  const int b = bh / H, h = bh - b * H;
  const int i = blockIdx.x * kPoolWaves + (threadIdx.x >> 6);
  if (i >= nb) return;  // uniform per wave
  const int lane = threadIdx.x & (kWave - 1);
  const int t0 = i * BLOCK;
  const int n_i = min(BLOCK, N - t0);
  const int c8 = lane & 15, r0 = lane >> 4;
  double acc[8];
  pool_sums<BLOCK>(x + b * st.b + h * st.h, st.n, t0, N, acc);
  double* o = out + ((int64_t)bh * nb + i) * kHeadDim + 8 * c8;
  if (r0 == 0) {
#pragma unroll
    for (int c = 0; c < 8; c += 2) *reinterpret_cast<f64x2*>(o + c) = (f64x2){acc[c], acc[c + 1]};
  }
  if (!is_k || split.frag == nullptr) return;  // uniform
  u32x4 whi, wlo;
  double sq;
  split_hi_lo(acc, whi, wlo, sq);
  if (r0 == 0) {
    const int64_t slot = (((int64_t)bh * split.ntiles + (i >> 5)) * kFSteps + (c8 >> 1)) * kWave +
                         (i & 31) + 32 * (c8 & 1);
    st16(split.frag + slot * 8, whi);
    st16(split.frag + (slot + 8 * kWave) * 8, wlo);
  }
  sq = row_sum16(sq);
  if (lane == 0) split.norm[(int64_t)bh * nb + i] = f32_round_up(sqrt(sq) / (double)n_i);
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

// The k largest of the wave's member keys (hi, lo words; ties to the lower
// index jj), written to out in ascending jj order.  Members must sit in
// ascending jj order over (slot t, lane).  Requires 1 <= k <= count(member).
template <int KPL>
__device__ __forceinline__ void select_emit(const uint32_t (&hi)[KPL], const uint32_t (&lo)[KPL],
                                            const bool (&member)[KPL], const int (&jj)[KPL],
                                            int k, int32_t* out) {
  bool exact;
  const uint32_t thi = kth_largest32<KPL>(hi, member, k, &exact);
  // selection: hi > thi, or hi == thi and (lo > tlo, or lo == tlo and among
  // the first need_eq such keys in index order)
  uint32_t tlo = 0;
  int need_eq = 0;
  if (!exact) {
    int gt = 0;
#pragma unroll
    for (int t = 0; t < KPL; ++t) gt += __popcll(__ballot(member[t] && hi[t] > thi));
    bool grp[KPL];
#pragma unroll
    for (int t = 0; t < KPL; ++t) grp[t] = member[t] && hi[t] == thi;
    bool ex2;
    tlo = kth_largest32<KPL>(lo, grp, k - gt, &ex2);
    int gt2 = 0;
#pragma unroll
    for (int t = 0; t < KPL; ++t) gt2 += __popcll(__ballot(grp[t] && lo[t] > tlo));
    need_eq = k - gt - gt2;
  }
  int taken = 0, eq_seen = 0;
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    bool sel;
    if (exact) {
      sel = member[t] && hi[t] >= thi;
    } else {
      const bool eq = member[t] && hi[t] == thi && lo[t] == tlo;
      const uint64_t eq_mask = __ballot(eq);
      const int eq_rank = eq_seen + rank_below(eq_mask);
      sel = (member[t] && (hi[t] > thi || (hi[t] == thi && lo[t] > tlo))) ||
            (eq && eq_rank < need_eq);
      eq_seen += __popcll(eq_mask);
    }
    const uint64_t sel_mask = __ballot(sel);
    if (sel) out[taken + rank_below(sel_mask)] = jj[t];
    taken += __popcll(sel_mask);
  }
}

// One wavefront per query block: the k largest of the row's order keys
// (64-bit), ties to the lower block index, emitted in ascending index order.
// Fast path: the k-th largest high word among the 64 lanes' maxima, P, bounds
// the row's k-th largest key from below (at least k keys have high word
// >= P), so only keys with high word >= P can be kept.  When at most 64 keys
// pass, they are compacted in index order, one per lane, and the exact
// selection runs on them; otherwise it runs on the whole row.  Either way the
// k-th largest key is found on its high 32 bits first; only the keys that tie
// with it there take part in the search over the low 32 bits.
template <int KPL>
__global__ __launch_bounds__(256) void topk_row_kernel(const double* __restrict__ scores,
                                                       int nb, int rows, int k_all, int kmax,
                                                       bool k_per_row, Shape cs,
                                                       int32_t* __restrict__ idx,
                                                       int32_t* __restrict__ cnt) {
  __shared__ uint32_t cand[4][3][kWave];  // per wave: candidate hi, lo, index
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = threadIdx.x >> 6;
  const int row = blockIdx.x * 4 + wv;
  if (row >= rows) return;  // uniform per wave
  // Candidate key blocks [jlo, jhi): under a causal window those holding an
  // allowed key of some query of the block (the allowed ranges never move
  // back as the query advances, so the first query's lower end and the last
  // query's upper end bound them); otherwise every block.
  int jlo = 0, jhi = nb;
  if (cs.causal_chunk > 0) {
    const int first = (row % nb) * cs.block;
    const int last = min(first + cs.block, cs.N) - 1;
    jlo = causal_lo(cs, first) / cs.block;
    jhi = (causal_hi(cs, last) + cs.block - 1) / cs.block;
  }
  // the row's k: one value for all rows, or (ragged mode) read from cnt;
  // never more than the candidates
  const int k = min(k_per_row ? __builtin_amdgcn_readfirstlane(cnt[row]) : k_all, jhi - jlo);
  const double* s = scores + (int64_t)row * nb;
  // Keys outside [jlo, jhi) are 0.  Every threshold below is >= 1 (a high
  // word of some lane's nonzero maximum), so they never pass a ">= P" test
  // and the fast path needs no separate membership flags.
  uint32_t hi[KPL], lo[KPL];
  int jj[KPL];
  uint32_t mhi = 0;  // high word of this lane's largest key (0: none)
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    const int j = lane + kWave * t;
    jj[t] = j;
    const uint64_t key = (j >= jlo && j < jhi) ? order_key(s[j]) : 0ull;
    hi[t] = (uint32_t)(key >> 32);
    lo[t] = (uint32_t)key;
    mhi = max(mhi, hi[t]);
  }
  int32_t* out = idx + (int64_t)row * kmax;

  bool fast = __popcll(__ballot(mhi != 0u)) >= k;
  uint32_t P = 0;
  int c = 0;
  if (fast) {  // wave-uniform
    const uint32_t mv[1] = {mhi};
    const bool mm[1] = {mhi != 0u};
    bool ex;
    P = kth_largest32<1>(mv, mm, k, &ex);
#pragma unroll
    for (int t = 0; t < KPL; ++t) c += __popcll(__ballot(hi[t] >= P));
    fast = c <= kWave;
  }
  if (fast) {
    // compact the candidates in ascending index order, one per lane
      int base = 0;
#pragma unroll
    for (int t = 0; t < KPL; ++t) {
      const bool ok = hi[t] >= P;
      const uint64_t m = __ballot(ok);
      if (ok) {
        const int pos = base + rank_below(m);
        cand[wv][0][pos] = hi[t];
        cand[wv][1][pos] = lo[t];
        cand[wv][2][pos] = (uint32_t)jj[t];
      }
      base += __popcll(m);
    }
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's writes landed
    __builtin_amdgcn_wave_barrier();
    const uint32_t ch[1] = {lane < c ? cand[wv][0][lane] : 0u};
    const uint32_t cl[1] = {lane < c ? cand[wv][1][lane] : 0u};
    const int cj[1] = {lane < c ? (int)cand[wv][2][lane] : 0};
    const bool cv[1] = {lane < c};
    select_emit<1>(ch, cl, cv, cj, k, out);
  } else {
    bool valid[KPL];
#pragma unroll
    for (int t = 0; t < KPL; ++t) valid[t] = jj[t] >= jlo && jj[t] < jhi;
    select_emit<KPL>(hi, lo, valid, jj, k, out);
  }
  for (int p = k + lane; p < kmax; p += kWave) out[p] = -1;
  if (lane == 0) cnt[row] = k;
}

template <int KPL>
hipError_t launch_topk(const double* scores, int nb, int rows, int k, int kmax, bool k_per_row,
                       const Shape& cs,
                       int32_t* idx, int32_t* cnt, hipStream_t stream) {
  topk_row_kernel<KPL><<<(rows + 3) / 4, 256, 0, stream>>>(scores, nb, rows, k, kmax, k_per_row,
                                                            cs, idx, cnt);
  return hipGetLastError();
}

// Row top-k over the score matrix with the register tile that fits nb.
hipError_t launch_topk_any(const double* scores, int nb, int rows, int k, int kmax,
                           bool k_per_row, const Shape& cs, int32_t* idx, int32_t* cnt,
                           hipStream_t stream) {
  const int kpl = (nb + kWave - 1) / kWave;
#define SA_TOPK(n) \
  if (kpl <= n) return launch_topk<n>(scores, nb, rows, k, kmax, k_per_row, cs, idx, cnt, stream);
  SA_TOPK(1) SA_TOPK(2) SA_TOPK(4) SA_TOPK(8) SA_TOPK(12) SA_TOPK(16) SA_TOPK(20) SA_TOPK(24)
  SA_TOPK(32)
#undef SA_TOPK
  return launch_topk<64>(scores, nb, rows, k, kmax, k_per_row, cs, idx, cnt, stream);
}

// ---- fused score + top-k (row mode) ---------------------------------------
// One workgroup of 8 waves per 32 query blocks of a (batch, head); scores for
// all nb key blocks stay in LDS as order-preserving 32-bit keys.
//
// Approximation.  With the pooled sums split as q = q1 + q2 + rq and
// k = k1 + k2 + rk (bf16 parts from the pooling, |rq| <= 2^-16 |q| (1 + 2^-14)
// per channel), a = (q1.k1 + q1.k2 + q2.k1) / (n_i n_j) is one chain of 24
// bf16 MFMAs (exact products, fp32 sums) and a multiply by the fp32
// reciprocal.  Per channel, the dropped terms q2 k2 + q1 rk + q2 rk + rq k are
// below 3.1 * 2^-16 |q_c k_c| (1 + 2^-7); the 384 products sum to at most
// 1.02 sum|q_c k_c|, and any order of 383 additions, each off by at most one
// fp32 ulp of its result, adds 383 * 2^-23 of that; the scaling adds 3 * 2^-24.
// In all |a - s| <= 9.5e-5 sum|q_c k_c| / (n_i n_j), and by Cauchy-Schwarz
// sum|q_c k_c| <= |q| |k|, so with qn = |q_i| / n_i and kn_max = max_j
// |k_j| / n_j (both rounded up by the pooling)
//     E = 2^-13 qn kn_max + 2^-120 (1 + qn n_i + kn_max block)
// bounds the error of every score of the row, the second term covering
// values the matrix cores flush to zero.  It holds while qn n_i and
// kn_max block stay below 2^60 (no fp32 overflow); other rows, and rows with
// non-finite inputs, take the exact path.  The fp64 scores of the other paths
// differ from s by ~1e-16 relative, far inside E.
//
// Classification.  With a_k, a_k1 the k-th and (k+1)-th largest
// approximations of the row, a key block with a > a_k1 + 2E outranks every
// block outside the k largest approximations, so it is among the k largest
// scores; one with a < a_k - 2E is below at least k scores and is dropped.
// The rest (the band) gets its exact fp64 score, and the k - (certain) best
// of the band under (score desc, index asc) are kept.  When the thresholds
// are compared as fp32 keys, they are rounded outwards.  The band is empty
// unless the gap between the k-th and (k+1)-th score is within 4E; a band of
// more than 64 blocks (heavy ties), an inconsistent count, or a row outside
// the bound's range takes the exact path: every candidate rescored in fp64
// and the selection of the unfused kernel run on the 64-bit keys.
constexpr int kFWaves = 8;
constexpr int kFThreads = kFWaves * kWave;
constexpr int kFStrideBig = 1192;   // LDS key-row stride = largest nb: 152.6 KB of keys
constexpr int kFStrideSmall = 584;  // 74.8 KB: two workgroups per CU
constexpr double kScoreRelErr = 1.0 / 8192;

// Order-preserving 32-bit key of an fp32 score (larger score -> larger key);
// -0 and +0 map to the same key; every finite score maps above 0.
__device__ __forceinline__ uint32_t order_key32(float a) {
  if (a == 0.f) a = 0.f;
  const uint32_t u = __float_as_uint(a);
  return (u >> 31) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key32_value(uint32_t key) {
  return __uint_as_float((key >> 31) ? (key ^ 0x80000000u) : ~key);
}

// fp64 score of one block pair from the pooled sums.
__device__ __forceinline__ double exact_score(const double* __restrict__ qrow,
                                              const double* __restrict__ krow, int nn) {
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll 4
  for (int c = 0; c < kHeadDim; c += 4) {
    const f64x2 a0 = *reinterpret_cast<const f64x2*>(qrow + c);
    const f64x2 a1 = *reinterpret_cast<const f64x2*>(qrow + c + 2);
    const f64x2 b0 = *reinterpret_cast<const f64x2*>(krow + c);
    const f64x2 b1 = *reinterpret_cast<const f64x2*>(krow + c + 2);
    acc[0] = fma(a0[0], b0[0], acc[0]);
    acc[1] = fma(a0[1], b0[1], acc[1]);
    acc[2] = fma(a1[0], b1[0], acc[2]);
    acc[3] = fma(a1[1], b1[1], acc[3]);
  }
  return ((acc[0] + acc[1]) + (acc[2] + acc[3])) / (double)nn;
}

// True for the lanes holding the `need` largest member keys (hi, lo words),
// ties to the lower lane.  Requires 1 <= need <= count(member).
__device__ __forceinline__ bool select_lanes(uint32_t hi, uint32_t lo, bool member, int need) {
  const uint32_t h[1] = {hi}, l[1] = {lo};
  const bool m[1] = {member};
  bool exact;
  const uint32_t thi = kth_largest32<1>(h, m, need, &exact);
  if (exact) return member && hi >= thi;
  const int gt = __popcll(__ballot(member && hi > thi));
  const bool grp[1] = {member && hi == thi};
  bool ex2;
  const uint32_t tlo = kth_largest32<1>(l, grp, need - gt, &ex2);
  const int gt2 = __popcll(__ballot(grp[0] && lo > tlo));
  const bool eq = grp[0] && lo == tlo;
  const int rank = rank_below(__ballot(eq));
  return (member && (hi > thi || (hi == thi && lo > tlo))) || (eq && rank < need - gt - gt2);
}

// Exact path of one row: every candidate in [jlo, jhi) rescored in fp64.
template <int KPL>
__device__ void exact_row_select(const double* __restrict__ qrow,
                                 const double* __restrict__ khead, const Shape& cs, int ni,
                                 int jlo, int jhi, int k, int32_t* out) {
  const int lane = threadIdx.x & (kWave - 1);
  uint32_t hi[KPL], lo[KPL];
  bool mem[KPL];
  int jj[KPL];
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    const int j = lane + kWave * t;
    jj[t] = j;
    mem[t] = j >= jlo && j < jhi;
    uint64_t key = 0ull;
    if (mem[t]) {
      const int nj = min(cs.block, cs.N - j * cs.block);
      key = order_key(exact_score(qrow, khead + (int64_t)j * kHeadDim, ni * nj));
    }
    hi[t] = (uint32_t)(key >> 32);
    lo[t] = (uint32_t)key;
  }
  select_emit<KPL>(hi, lo, mem, jj, k, out);
}

template <int NBP, int BLOCK>
__global__ __launch_bounds__(kFThreads) void score_topk_kernel(
    const uint16_t* __restrict__ q, Strides qs, const uint16_t* __restrict__ kfrag,
    const float* __restrict__ knorm, double* __restrict__ qhat, const double* __restrict__ khat,
    Shape cs, int k_all, int kmax, int ntiles, int per_xcd, int32_t* __restrict__ idx,
    int32_t* __restrict__ cnt) {
  constexpr int KPL = (NBP + kWave - 1) / kWave;
  static_assert(NBP % 4 == 0 && NBP >= 129, "a key row holds one parked query block, 16-byte aligned");
  __shared__ __align__(16) uint32_t keys[kFRows * NBP];
  __shared__ uint32_t cand[kFWaves][2][kWave];
  __shared__ float wmax[kFWaves];
  const int nb = cs.nb;
  constexpr int kQB = kFRows / kFWaves;  // query blocks pooled per wave
  // Consecutive tiles (the same head's key blocks) run on one XCD: workgroup
  // w goes to XCD w % 8, which takes the logical tiles [x, x + 1) * per_xcd.
  const int logical = (int)(blockIdx.x & 7) * per_xcd + (int)(blockIdx.x >> 3);
  if (logical >= cs.B * cs.H * ntiles) return;  // uniform
  const int bh = logical / ntiles, it = logical - bh * ntiles;
  const int lane = threadIdx.x & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int l32 = lane & 31, g = lane >> 5;
  const int c8 = lane & 15, r0 = lane >> 4;

  // The head's key norms, read ahead of the pooling (a clamped index repeats
  // a norm, which does not change their max).
  constexpr int kKnLoads = (NBP + kFThreads - 1) / kFThreads;
  float kv[kKnLoads];
#pragma unroll
  for (int u = 0; u < kKnLoads; ++u)
    kv[u] = knorm[(int64_t)bh * nb + min((int)threadIdx.x + kFThreads * u, nb - 1)];

  // Query pooling (the same arithmetic as the K pooling): wave w pools the
  // tile's query blocks kQB w + u.  The fp64 sums go to qhat for the
  // rescoring paths; the hi/lo operand words and the norm are parked in the
  // key area (not in use yet), block kQB w + u in key row w + kFWaves u (hi
  // words of channels 8 c .. 8 c + 7 at word 4 c, lo words at 64 + 4 c, the
  // norm at 128).  Blocks past nb pool to zero.
  const uint16_t* qhead = q + (bh / cs.H) * qs.b + (bh % cs.H) * qs.h;
  auto park = [&](const double (&acc)[8], int u) __attribute__((always_inline)) {
    const int i = it * kFRows + kQB * wave + u;
    if (i < nb && r0 == 0) {
      double* o = qhat + ((int64_t)bh * nb + i) * kHeadDim + 8 * c8;
#pragma unroll
      for (int c = 0; c < 8; c += 2) *reinterpret_cast<f64x2*>(o + c) = (f64x2){acc[c], acc[c + 1]};
    }
    u32x4 whi, wlo;
    double sq;
    split_hi_lo(acc, whi, wlo, sq);
    uint32_t* slot = keys + (wave + kFWaves * u) * NBP;
    if (r0 == 0) {
      *reinterpret_cast<u32x4*>(slot + 4 * c8) = whi;
      *reinterpret_cast<u32x4*>(slot + 64 + 4 * c8) = wlo;
    }
    sq = row_sum16(sq);
    const int n_i = min(cs.block, cs.N - i * cs.block);
    if (lane == 0) slot[128] = __float_as_uint(n_i > 0 ? f32_round_up(sqrt(sq) / (double)n_i) : 0.f);
  };
  {  // BLOCK 64: two blocks' loads in flight together
    constexpr int kPar = BLOCK == 64 ? 2 : 1;
#pragma unroll
    for (int u0 = 0; u0 < kQB; u0 += kPar) {
      u32x4 w[kPar][BLOCK / 4];
#pragma unroll
      for (int p = 0; p < kPar; ++p)
        pool_load<BLOCK>(qhead, qs.n, (it * kFRows + kQB * wave + u0 + p) * BLOCK, cs.N, w[p]);
#pragma unroll
      for (int p = 0; p < kPar; ++p) {
        double acc[8];
        pool_reduce<BLOCK>(w[p], (it * kFRows + kQB * wave + u0 + p) * BLOCK, cs.N, acc);
        park(acc, u0 + p);
      }
    }
  }

  // kn_max of the head (a non-finite norm makes it +inf)
  float m = 0.f;
#pragma unroll
  for (int u = 0; u < kKnLoads; ++u)
    m = kv[u] <= 3.4028235e38f ? fmaxf(m, kv[u]) : __builtin_huge_valf();
  m = wave_max(m);
  if (lane == 0) wmax[wave] = m;
  __syncthreads();
  // qn of this wave's rows wave + 8 m (lane m): block rr parked in key row
  // rr / kQB + kFWaves (rr % kQB)
  float qn_rows = 0.f;
  if (lane < kQB) {
    const int rr = wave + kFWaves * lane;
    qn_rows = __uint_as_float(keys[(rr / kQB + kFWaves * (rr % kQB)) * NBP + 128]);
  }

  {  // approximate scores of the 32 query blocks against every key block
    // operand step st, lane l: channels 8 (2 (st % 8) + l / 32) .. +7 of
    // query block l % 32, hi words for st < 8, lo words after
    bf16x8 qa[kFSteps];
    {
      const int rb = l32;
      const uint32_t* src = keys + (rb / kQB + kFWaves * (rb % kQB)) * NBP + 4 * g;
#pragma unroll
      for (int st = 0; st < kFSteps; ++st)
        qa[st] = __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(src + (st < 8 ? 0 : 64) + 8 * (st & 7)));
    }
    __syncthreads();  // every wave holds its operands before the keys overwrite them
    const u32x4* ksrc =
        reinterpret_cast<const u32x4*>(kfrag) + (int64_t)bh * ntiles * kFSteps * kWave + lane;
    auto load = [&](bf16x8 (&kb)[kFSteps], int jt) {
#pragma unroll
      for (int st = 0; st < kFSteps; ++st)
        kb[st] = __builtin_bit_cast(bf16x8, ksrc[((int64_t)jt * kFSteps + st) * kWave]);
    };
    auto products = [&](const bf16x8 (&kb)[kFSteps]) {
      f32x16 acc = {};
#pragma unroll
      for (int st = 0; st < 8; ++st)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[8 + st], kb[st], acc, 0, 0, 0);
#pragma unroll
      for (int st = 0; st < 8; ++st)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[st], kb[8 + st], acc, 0, 0, 0);
#pragma unroll
      for (int st = 0; st < 8; ++st)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[st], kb[st], acc, 0, 0, 0);
      return acc;
    };
    // Keys of a tile: lane holds key block j, query blocks 8 (r / 4) + 4 g +
    // r % 4 of the tile (rows past nb are written but never read).  Every
    // query block is scaled as if it held `block` tokens: only the last one
    // can be shorter, and a common factor of its row keeps its order (its
    // error bound is scaled by the same factor).  fma(.., +0) turns -0 to +0.
    auto store_keys = [&](const f32x16& acc, int jt) {
      const int j = jt * 32 + l32;
      if (j < nb) {
        const float inv =
            __builtin_amdgcn_rcpf((float)(cs.block * min(cs.block, cs.N - j * cs.block)));
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t u = __float_as_uint(fmaf(acc[r], inv, 0.f));
          keys[(8 * (r >> 2) + 4 * g + (r & 3)) * NBP + j] =
              u ^ ((uint32_t)((int32_t)u >> 31) | 0x80000000u);
        }
      }
    };
    // Two operand buffers: the next tile's loads are in flight during the
    // current tile's products, and the previous tile's keys are stored while
    // the current tile's products run.  The loads are unconditional (clamped
    // to the last tile) so that the waits before the products count only the
    // current tile's.
    bf16x8 ka[kFSteps], kc[kFSteps];
    f32x16 prev = {};
    int jprev = -1;
    load(ka, min(wave, ntiles - 1));
    for (int jt = wave; jt < ntiles; jt += 2 * kFWaves) {
      load(kc, min(jt + kFWaves, ntiles - 1));
      __builtin_amdgcn_sched_barrier(0);
      f32x16 cur = products(ka);
      if (jprev >= 0) store_keys(prev, jprev);
      prev = cur;
      jprev = jt;
      __builtin_amdgcn_sched_barrier(0);
      load(ka, min(jt + 2 * kFWaves, ntiles - 1));
      __builtin_amdgcn_sched_barrier(0);
      if (jt + kFWaves < ntiles) {
        cur = products(kc);
        store_keys(prev, jprev);
        prev = cur;
        jprev = jt + kFWaves;
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if (jprev >= 0) store_keys(prev, jprev);
  }
  __syncthreads();
  float kn_max = wmax[0];
#pragma unroll
  for (int w = 1; w < kFWaves; ++w) kn_max = fmaxf(kn_max, wmax[w]);
  const double* khead = khat + (int64_t)bh * nb * kHeadDim;
  uint32_t* ckey = cand[wave][0];
  uint32_t* cidx = cand[wave][1];

  for (int rm = 0; rm < kQB; ++rm) {
    const int rr = wave + kFWaves * rm;
    const int i = it * kFRows + rr;
    if (i >= nb) break;  // uniform
    const int64_t row = (int64_t)bh * nb + i;
    const int ni = min(cs.block, cs.N - i * cs.block);
    // candidate key blocks, as in the unfused row top-k
    int jlo = 0, jhi = nb;
    if (cs.causal_chunk > 0) {
      const int first = i * cs.block;
      const int last = min(first + cs.block, cs.N) - 1;
      jlo = causal_lo(cs, first) / cs.block;
      jhi = (causal_hi(cs, last) + cs.block - 1) / cs.block;
    }
    const int k = min(k_all, jhi - jlo);
    int32_t* out = idx + row * kmax;
    const double* qrow = qhat + row * kHeadDim;
    const float qn = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(qn_rows), rm));
    // the keys of a short last row are scaled by ni / block, and so is E
    const double E = (kScoreRelErr * (double)qn * (double)kn_max +
                      0x1p-120 * (1.0 + (double)qn * ni + (double)kn_max * cs.block)) *
                     ((double)ni / cs.block);
    const bool bounded = (double)qn * ni <= 0x1p60 && (double)kn_max * cs.block <= 0x1p60;
    // keys of a_k - 2E rounded down and a_k1 + 2E rounded up
    uint32_t KLO = 0, KHI = 0;
    auto thresholds = [&](uint32_t kk, uint32_t kk1) {
      const double lo = (double)key32_value(kk) - 2.0 * E;
      const double hi = (double)key32_value(kk1) + 2.0 * E;
      const float flo = (float)lo, fhi = (float)hi;
      KLO = order_key32(flo) - ((double)flo > lo ? 1u : 0u);
      KHI = order_key32(fhi) + ((double)fhi < hi ? 1u : 0u);
    };
    if (k >= jhi - jlo) {
      for (int p = lane; p < k; p += kWave) out[p] = jlo + p;
    } else if (!bounded) {
      exact_row_select<KPL>(qrow, khead, cs, ni, jlo, jhi, k, out);
    } else {
      uint32_t key[KPL];
      uint32_t mk = 0;  // 0: not a candidate (below every score's key)
#pragma unroll
      for (int t = 0; t < KPL; ++t)  // every read issued (clamped into the row)
        key[t] = keys[rr * NBP + min(lane + kWave * t, NBP - 1)];
#pragma unroll
      for (int t = 0; t < KPL; ++t) {
        // opaque to the compiler, which would otherwise turn the select below
        // into a branch around each read and wait on each one
        asm volatile("" : "+v"(key[t]));
        const int j = lane + kWave * t;
        key[t] = (j >= jlo && j < jhi) ? key[t] : 0u;
        mk = max(mk, key[t]);
      }
      // As in the unfused kernel, the k-th largest lane maximum P bounds the
      // k-th key from below; the keys >= P are compacted in index order.
      bool done = false, have = false;
      const bool enough = __popcll(__ballot(mk != 0u)) >= k;
      uint32_t P = 0;
      int c = 0;
      if (enough) {
        const uint32_t mv[1] = {mk};
        const bool mm[1] = {mk != 0u};
        bool ex;
        P = kth_largest32<1>(mv, mm, k, &ex);
#pragma unroll
        for (int t = 0; t < KPL; ++t) {
          const bool ok = key[t] >= P;
          const uint64_t m = __ballot(ok);
          const int pos = c + rank_below(m);
          if (ok && pos < kWave) {
            ckey[pos] = key[t];
            cidx[pos] = (uint32_t)(lane + kWave * t);
          }
          c += __popcll(m);
        }
      }
      if (enough && c <= kWave) {
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's writes landed
        __builtin_amdgcn_wave_barrier();
        const bool cm = lane < c;
        const uint32_t ck = cm ? ckey[lane] : 0u;
        const int cj = cm ? (int)cidx[lane] : 0;
        const uint32_t cv[1] = {ck};
        const bool cmm[1] = {cm};
        bool ex;
        // below P only when exactly k keys are >= P: then P itself separates them
        const uint32_t T = max(kth_largest32<1>(cv, cmm, k, &ex), P);
        // a_k and a_k1: the extremes on either side of T, or T itself when it
        // is tied across the k-th place
        uint32_t kk = T, kk1 = T;
        if (__popcll(__ballot(cm && ck >= T)) == k) {
          kk = wave_min_u32(cm && ck >= T ? ck : ~0u);
          if (c > k) {
            kk1 = wave_max_u32(cm && ck < T ? ck : 0u);
          } else {  // the (k+1)-th key is the row's largest below P
            uint32_t mx = 0u;
#pragma unroll
            for (int t = 0; t < KPL; ++t) mx = max(mx, key[t] < P ? key[t] : 0u);
            kk1 = wave_max_u32(mx);
          }
        }
        thresholds(kk, kk1);
        have = true;
        // empty band: the k keys above KHI are all among the candidates
        const bool sel = cm && ck > KHI;
        const uint64_t m = __ballot(sel);
        if (KLO > KHI && __popcll(m) == k) {
          if (sel) out[rank_below(m)] = cj;
          done = true;
        } else if (KLO >= P) {
          // Every key >= KLO is >= P, hence a candidate: the band is the
          // candidates in [KLO, KHI].  Each band block is rescored in fp64 by
          // the whole wave (lane l: channels 2 l, 2 l + 1), its 64-bit key
          // kept by the candidate's lane; the k - (certain) best band lanes
          // then join the certain ones, all in index order.
          const bool band = cm && ck >= KLO && ck <= KHI;
          const uint64_t bm = __ballot(band);
          const int cin = __popcll(m), cband = __popcll(bm);
          if (cin <= k && cin + cband >= k) {
            const f64x2 qv = *reinterpret_cast<const f64x2*>(qrow + 2 * lane);
            uint32_t bhi = 0u, blo = 0u;
            uint64_t rest = bm;
            while (rest != 0ull) {  // uniform; four blocks' loads in flight
              int lm[4];
              int last = 0;
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                if (rest != 0ull) {
                  last = (int)__builtin_ctzll(rest);
                  rest &= rest - 1ull;
                }
                lm[u] = last;
              }
              f64x2 kv[4];
              int jm[4];
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                jm[u] = __builtin_amdgcn_readlane(cj, lm[u]);
                kv[u] = *reinterpret_cast<const f64x2*>(khead + (int64_t)jm[u] * kHeadDim + 2 * lane);
              }
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                const double d = wave_sum_f64(fma(qv[0], kv[u][0], qv[1] * kv[u][1]));
                const int nj = min(cs.block, cs.N - jm[u] * cs.block);
                const uint64_t k64 = order_key(d / (double)(ni * nj));
                if (lane == lm[u]) {
                  bhi = (uint32_t)(k64 >> 32);
                  blo = (uint32_t)k64;
                }
              }
            }
            const bool sb = cin < k ? select_lanes(bhi, blo, band, k - cin) : false;
            const bool keep = sel || sb;
            const uint64_t km = __ballot(keep);
            if (keep) out[rank_below(km)] = cj;
            done = true;
          }
        }
      }
      if (!done) {
        if (!have) {
          bool mem[KPL];
#pragma unroll
          for (int t = 0; t < KPL; ++t) mem[t] = key[t] != 0u;
          bool ex;
          const uint32_t T = kth_largest32<KPL>(key, mem, k, &ex);
          int cge = 0;
          uint32_t mn = ~0u, mx = 0u;
#pragma unroll
          for (int t = 0; t < KPL; ++t) {
            const bool ge = key[t] >= T && key[t] != 0u;
            cge += __popcll(__ballot(ge));
            if (ge) mn = min(mn, key[t]);
            else mx = max(mx, key[t]);
          }
          if (cge == k) thresholds(wave_min_u32(mn), wave_max_u32(mx));
          else thresholds(T, T);
        }
        int cin = 0, cband = 0;
#pragma unroll
        for (int t = 0; t < KPL; ++t) {
          cin += __popcll(__ballot(key[t] > KHI));
          cband += __popcll(__ballot(key[t] != 0u && key[t] <= KHI && key[t] >= KLO));
        }
        if (cband <= kWave && cin <= k && cin + cband >= k) {
          // compact the band's indices; rescore them in fp64, all lanes on
          // one block at a time (lane l: channels 2 l, 2 l + 1)
          int base = 0;
#pragma unroll
          for (int t = 0; t < KPL; ++t) {
            const bool b = key[t] != 0u && key[t] <= KHI && key[t] >= KLO;
            const uint64_t m = __ballot(b);
            if (b) cidx[base + rank_below(m)] = (uint32_t)(lane + kWave * t);
            base += __popcll(m);
          }
          __builtin_amdgcn_s_waitcnt(0xC07F);
          __builtin_amdgcn_wave_barrier();
          const f64x2 qv = *reinterpret_cast<const f64x2*>(qrow + 2 * lane);
          uint32_t bhi = 0u, blo = 0u;
          for (int m0 = 0; m0 < cband; m0 += 4) {  // uniform
            f64x2 kv[4];
            int jm[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              jm[u] = (int)cidx[min(m0 + u, cband - 1)];
              kv[u] = *reinterpret_cast<const f64x2*>(khead + (int64_t)jm[u] * kHeadDim + 2 * lane);
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const double d = wave_sum_f64(fma(qv[0], kv[u][0], qv[1] * kv[u][1]));
              const int nj = min(cs.block, cs.N - jm[u] * cs.block);
              const uint64_t k64 = order_key(d / (double)(ni * nj));
              if (lane == m0 + u) {
                bhi = (uint32_t)(k64 >> 32);
                blo = (uint32_t)k64;
              }
            }
          }
          const bool sel_band = cin < k && select_lanes(bhi, blo, lane < cband, k - cin);
          ckey[lane] = sel_band ? 1u : 0u;
          __builtin_amdgcn_s_waitcnt(0xC07F);
          __builtin_amdgcn_wave_barrier();
          int taken = 0;
          base = 0;
#pragma unroll
          for (int t = 0; t < KPL; ++t) {
            const bool b = key[t] != 0u && key[t] <= KHI && key[t] >= KLO;
            const uint64_t bmask = __ballot(b);
            const bool sel = key[t] > KHI || (b && ckey[base + rank_below(bmask)] != 0u);
            base += __popcll(bmask);
            const uint64_t m = __ballot(sel);
            const int pos = taken + rank_below(m);
            if (sel && pos < k) out[pos] = lane + kWave * t;
            taken += __popcll(m);
          }
        } else {
          exact_row_select<KPL>(qrow, khead, cs, ni, jlo, jhi, k, out);
        }
      }
    }
    for (int p = k + lane; p < kmax; p += kWave) out[p] = -1;
    if (lane == 0) cnt[row] = k;
    // (the next row rewrites this wave's cand slots: a wave's LDS accesses
    // complete in order, so the reads above see this row's values)
  }
}

// ---- whole-head ragged selection ------------------------------------------
// Per (batch, head): every query block keeps its best key block; the other
// (budget - nqb) pairs are the largest of the remaining ones under (score
// desc, i asc, j asc).  Within a row, the pairs so kept are always a prefix of
// the row's own order (score desc, j asc), so the mode reduces to a per-row
// count c_i followed by the row top-k with k_i = min(c_i, kmax):
//   top1   : each row's best key block (excluded from the global ranking)
//   radix  : the (budget - nqb)-th largest order key T among the remaining
//            pairs, by 8 passes of 8 bits (a 256-bin histogram, then one
//            workgroup per head picks the digit), and the number r of pairs
//            equal to T that are kept (those first in (i, j) order)
//   counts : per row, remaining pairs with key > T and with key == T
//   row k  : c_i = 1 + above_i + clamp(r - (ties in rows < i), 0, ties_i)
struct HeadState {
  unsigned long long prefix;  // radix prefix; T after the last pass
  long long need;             // rank still to find among the keys == prefix
  int none;                   // no pair beyond the row bests is kept
  int pad[3];
};
constexpr int kBins = 256;

struct HeadWs {
  HeadState* st;    // [BH]
  uint32_t* hist;   // [BH][256]
  int32_t* top1;    // [rows]
  int32_t* above;   // [rows]
  int32_t* ties;    // [rows]
};

__global__ __launch_bounds__(kBins) void head_init_kernel(HeadWs w, long long rest) {
  const int bh = blockIdx.x;
  w.hist[bh * kBins + threadIdx.x] = 0u;
  if (threadIdx.x == 0) {
    w.st[bh].prefix = 0ull;
    w.st[bh].need = rest;
    w.st[bh].none = rest == 0;
  }
}

// One wave per row: the largest key, lowest index first.
__global__ __launch_bounds__(256) void row_top1_kernel(const double* __restrict__ scores, int nb,
                                                       int rows, int32_t* __restrict__ top1) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const double* s = scores + (int64_t)row * nb;
  uint64_t best = 0ull;  // below every finite score
  int bj = nb;
  for (int j = lane; j < nb; j += kWave) {
    const uint64_t key = order_key(s[j]);
    if (key > best) {  // ascending j within the lane: ties keep the first
      best = key;
      bj = j;
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const uint64_t ok = __shfl_xor(best, o, kWave);
    const int oj = __shfl_xor(bj, o, kWave);
    if (ok > best || (ok == best && oj < bj)) {
      best = ok;
      bj = oj;
    }
  }
  if (lane == 0) top1[row] = bj;
}

// Histogram of the next 8-bit digit (bits shift..shift+7) of the order keys
// of the remaining pairs that match the prefix found so far.  Blocks of 4
// rows; equal digits of a wave are counted with one ballot and one LDS add.
__global__ __launch_bounds__(256) void head_hist_kernel(const double* __restrict__ scores, int nb,
                                                        HeadWs w, int shift) {
  __shared__ uint32_t h[kBins];
  const int bh = blockIdx.y;
  if (w.st[bh].none) return;  // uniform per workgroup
  const uint64_t prefix = w.st[bh].prefix;
  const uint64_t mask = shift == 56 ? 0ull : ~0ull << (shift + 8);
  h[threadIdx.x] = 0u;
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (i < nb) {
    const int64_t row = (int64_t)bh * nb + i;
    const double* s = scores + row * nb;
    const int skip = w.top1[row];
    for (int j0 = 0; j0 < nb; j0 += kWave) {
      const int j = j0 + lane;
      bool act = false;
      uint32_t bin = 0;
      if (j < nb && j != skip) {
        const uint64_t key = order_key(s[j]);
        act = (key & mask) == (prefix & mask);
        bin = (uint32_t)(key >> shift) & (kBins - 1);
      }
      uint64_t left = __ballot(act);
      while (left) {
        const int first = __ffsll((long long)left) - 1;
        const uint32_t b = __shfl(bin, first, kWave);
        const uint64_t same = __ballot(act && bin == b);
        if (lane == first) atomicAdd(&h[b], (uint32_t)__popcll(same));
        left &= ~same;
        if (act && bin == b) act = false;
      }
    }
  }
  __syncthreads();
  const uint32_t c = h[threadIdx.x];
  if (c) atomicAdd(&w.hist[bh * kBins + threadIdx.x], c);
}

// One workgroup per head: the digit that holds the need-th largest key,
// scanning bins from the top; clears the histogram for the next pass.
__global__ __launch_bounds__(kBins) void head_radix_step_kernel(HeadWs w, int shift) {
  __shared__ uint32_t wsum[kBins / kWave];
  const int bh = blockIdx.x, t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int d = kBins - 1 - t;  // thread t holds bin d: t ascending = digit descending
  const uint32_t c = w.hist[bh * kBins + d];
  w.hist[bh * kBins + d] = 0u;
  if (w.st[bh].none) return;  // uniform per workgroup
  uint32_t incl = c;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += y;
  }
  if (lane == kWave - 1) wsum[wave] = incl;
  __syncthreads();
  for (int v = 0; v < wave; ++v) incl += wsum[v];
  const long long need = w.st[bh].need;
  const long long excl = (long long)incl - c;  // keys in higher digits
  __syncthreads();
  if (c > 0 && excl < need && (long long)incl >= need) {
    w.st[bh].prefix |= (unsigned long long)d << shift;
    w.st[bh].need = need - excl;
  }
}

// One wave per row: remaining pairs above and equal to the threshold key.
__global__ __launch_bounds__(256) void head_count_kernel(const double* __restrict__ scores, int nb,
                                                         int rows, HeadWs w) {
  const int lane = threadIdx.x & (kWave - 1);
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int bh = row / nb;
  int above = 0, ties = 0;
  if (!w.st[bh].none) {
    const uint64_t T = w.st[bh].prefix;
    const double* s = scores + (int64_t)row * nb;
    const int skip = w.top1[row];
    for (int j0 = 0; j0 < nb; j0 += kWave) {
      const int j = j0 + lane;
      uint64_t key = 0ull;
      if (j < nb && j != skip) key = order_key(s[j]);
      above += __popcll(__ballot(key > T));
      ties += __popcll(__ballot(key == T && key != 0ull));
    }
  }
  if (lane == 0) {
    w.above[row] = above;
    w.ties[row] = ties;
  }
}

// One workgroup per head: the ties at T are kept first in row order, so row i
// keeps clamp(r - ties in earlier rows, 0, ties_i) of them.  Writes each row's
// k = min(c_i, kmax) into cnt (read back by the row top-k).
constexpr int kRowKThreads = 1024;
__global__ __launch_bounds__(kRowKThreads) void head_rowk_kernel(int nb, int kmax, HeadWs w,
                                                                 int32_t* __restrict__ cnt) {
  __shared__ long long wsum[kRowKThreads / kWave];
  __shared__ long long carry;
  const int bh = blockIdx.x, t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const long long r = w.st[bh].none ? 0 : w.st[bh].need;
  if (t == 0) carry = 0;
  __syncthreads();
  for (int i0 = 0; i0 < nb; i0 += kRowKThreads) {
    const int i = i0 + t;
    const int64_t row = (int64_t)bh * nb + i;
    const long long e = i < nb ? w.ties[row] : 0;
    long long incl = e;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const long long y = __shfl_up(incl, o, kWave);
      if (lane >= o) incl += y;
    }
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    long long before = carry + incl - e;
    for (int v = 0; v < wave; ++v) before += wsum[v];
    if (i < nb) {
      const long long take = min(max(r - before, 0ll), e);
      const long long c = 1 + (long long)w.above[row] + take;
      cnt[row] = (int32_t)min(c, (long long)kmax);
    }
    __syncthreads();
    if (t == 0) {
      long long tot = 0;
      for (int v = 0; v < kRowKThreads / kWave; ++v) tot += wsum[v];
      carry += tot;
    }
    __syncthreads();
  }
}

}  // namespace

// Pools Q and K (k_only: K alone).
static void launch_pool(const Shape& s, const void* q, Strides qs, const void* k, Strides ks,
                        double* qhat, double* khat, const PoolSplit& sp, bool k_only,
                        hipStream_t stream) {
  const dim3 grid((s.nb + kPoolWaves - 1) / kPoolWaves, (unsigned)(s.B * s.H), k_only ? 1 : 2);
  const int z0 = k_only ? 1 : 0;
  const auto* qq = static_cast<const uint16_t*>(q);
  const auto* kk = static_cast<const uint16_t*>(k);
  if (s.block == 64)
    pool_kernel<64><<<grid, kPoolWaves * kWave, 0, stream>>>(qq, kk, qs, ks, s.H, s.N, s.nb, z0,
                                                             qhat, khat, sp);
  else
    pool_kernel<128><<<grid, kPoolWaves * kWave, 0, stream>>>(qq, kk, qs, ks, s.H, s.N, s.nb, z0,
                                                              qhat, khat, sp);
}

// Row mode: pooled sums, then either the fused path's split operands and
// norms (nb <= kFStrideBig) or the score matrix.
size_t select_workspace_bytes(const Shape& s) {
  const size_t bh = (size_t)s.B * s.H;
  const size_t pooled = bh * s.nb * kHeadDim * sizeof(double) * 2;
  if (s.nb <= kFStrideBig) {
    const size_t ntiles = (s.nb + kFRows - 1) / kFRows;
    return pooled + bh * ntiles * kFSteps * kWave * 8 * sizeof(uint16_t) +
           bh * s.nb * sizeof(float);
  }
  return pooled + bh * s.nb * s.nb * sizeof(double);
}

// Whole-head mode: pooled sums, the score matrix and the radix-select state.
size_t select_head_workspace_bytes(const Shape& s) {
  const size_t bh = (size_t)s.B * s.H;
  const size_t rows = bh * s.nb;
  return bh * s.nb * kHeadDim * sizeof(double) * 2 + bh * s.nb * s.nb * sizeof(double) +
         bh * sizeof(HeadState) + bh * kBins * sizeof(uint32_t) + 3 * rows * sizeof(int32_t);
}

static hipError_t launch_pool_score(const Shape& s, const void* q, Strides qs, const void* k,
                                    Strides ks, void* ws, double** scores_out,
                                    hipStream_t stream) {
  const size_t bh = (size_t)s.B * s.H;
  double* qhat = static_cast<double*>(ws);
  double* khat = qhat + bh * s.nb * kHeadDim;
  double* scores = khat + bh * s.nb * kHeadDim;
  launch_pool(s, q, qs, k, ks, qhat, khat, PoolSplit{}, false, stream);
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
  if (s.nb <= kFStrideBig) {
    const size_t bh = (size_t)s.B * s.H;
    const int ntiles = (s.nb + kFRows - 1) / kFRows;
    const size_t frag = bh * ntiles * kFSteps * kWave * 8;  // uint16
    double* qhat = static_cast<double*>(ws);
    double* khat = qhat + bh * s.nb * kHeadDim;
    PoolSplit sp;
    sp.frag = reinterpret_cast<uint16_t*>(khat + bh * s.nb * kHeadDim);
    sp.norm = reinterpret_cast<float*>(sp.frag + frag);
    sp.ntiles = ntiles;
    // K alone: every workgroup of the fused kernel pools its own query blocks
    launch_pool(s, q, qs, k, ks, qhat, khat, sp, true, stream);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int per_xcd = (int)((bh * ntiles + 7) / 8);
    const auto* qq = static_cast<const uint16_t*>(q);
#define SA_FUSED(NBP, BLOCK)                                                                   \
  score_topk_kernel<NBP, BLOCK><<<8 * per_xcd, kFThreads, 0, stream>>>(                         \
      qq, qs, sp.frag, sp.norm, qhat, khat, s, topk, kmax, ntiles, per_xcd, idx, cnt)
    if (s.nb <= kFStrideSmall) {
      if (s.block == 64) SA_FUSED(kFStrideSmall, 64);
      else SA_FUSED(kFStrideSmall, 128);
    } else {
      if (s.block == 64) SA_FUSED(kFStrideBig, 64);
      else SA_FUSED(kFStrideBig, 128);
    }
#undef SA_FUSED
    return hipGetLastError();
  }
  double* scores = nullptr;
  hipError_t e = launch_pool_score(s, q, qs, k, ks, ws, &scores, stream);
  if (e != hipSuccess) return e;
  const int rows = s.B * s.H * s.nb;
  return launch_topk_any(scores, s.nb, rows, topk, kmax, false, s, idx, cnt, stream);
}

hipError_t launch_select_head(const Shape& s, const void* q, Strides qs, const void* k,
                              Strides ks, int64_t budget, int kmax, int32_t* idx, int32_t* cnt,
                              void* ws, hipStream_t stream) {
  double* scores = nullptr;
  hipError_t e = launch_pool_score(s, q, qs, k, ks, ws, &scores, stream);
  if (e != hipSuccess) return e;
  const int bh = s.B * s.H;
  const int rows = bh * s.nb;
  HeadWs w;
  w.st = reinterpret_cast<HeadState*>(scores + (size_t)rows * s.nb);
  w.hist = reinterpret_cast<uint32_t*>(w.st + bh);
  w.top1 = reinterpret_cast<int32_t*>(w.hist + (size_t)bh * kBins);
  w.above = w.top1 + rows;
  w.ties = w.above + rows;
  head_init_kernel<<<bh, kBins, 0, stream>>>(w, (long long)(budget - s.nb));
  row_top1_kernel<<<(rows + 3) / 4, 256, 0, stream>>>(scores, s.nb, rows, w.top1);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  for (int shift = 56; shift >= 0; shift -= 8) {
    head_hist_kernel<<<dim3((s.nb + 3) / 4, bh), 256, 0, stream>>>(scores, s.nb, w, shift);
    head_radix_step_kernel<<<bh, kBins, 0, stream>>>(w, shift);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  head_count_kernel<<<(rows + 3) / 4, 256, 0, stream>>>(scores, s.nb, rows, w);
  head_rowk_kernel<<<bh, kRowKThreads, 0, stream>>>(s.nb, kmax, w, cnt);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  Shape unrestricted = s;  // the whole-head mode has no causal window
  unrestricted.causal_chunk = 0;
  unrestricted.causal_window = 0;
  return launch_topk_any(scores, s.nb, rows, 0, kmax, true, unrestricted, idx, cnt, stream);
}

}  // namespace sa

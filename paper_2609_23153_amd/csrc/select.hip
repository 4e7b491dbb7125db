// Block selection M_phi on gfx950 (paper §2 Eq. comp-sparse; selection kept
// in BF16 inputs per §4.3): mean-pooled block scores and per-query-block
// top-k with ties to the lower block index, or the ragged whole-head variant.
//
// Launches:
//   pool   : Q and K streamed once from HBM; per block, the fp64 sum of the
//            bf16 token vectors (exact for bf16 inputs whose exponents span
//            fewer than ~38 binades, so it does not depend on summation order)
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
  const uint64_t below = lanes_below_mask();
  int taken = 0, eq_seen = 0;
#pragma unroll
  for (int t = 0; t < KPL; ++t) {
    bool sel;
    if (exact) {
      sel = member[t] && hi[t] >= thi;
    } else {
      const bool eq = member[t] && hi[t] == thi && lo[t] == tlo;
      const uint64_t eq_mask = __ballot(eq);
      const int eq_rank = eq_seen + __popcll(eq_mask & below);
      sel = (member[t] && (hi[t] > thi || (hi[t] == thi && lo[t] > tlo))) ||
            (eq && eq_rank < need_eq);
      eq_seen += __popcll(eq_mask);
    }
    const uint64_t sel_mask = __ballot(sel);
    if (sel) out[taken + __popcll(sel_mask & below)] = jj[t];
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
    const uint64_t below = lanes_below_mask();
    int base = 0;
#pragma unroll
    for (int t = 0; t < KPL; ++t) {
      const bool ok = hi[t] >= P;
      const uint64_t m = __ballot(ok);
      if (ok) {
        const int pos = base + __popcll(m & below);
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

size_t select_workspace_bytes(const Shape& s) {
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

// Fused block-sparse attention forward on fp8 (OCP e4m3) operands, gfx950.
//
// The same result as the bf16 forward (paper §2 Eq. comp-sparse, §4.1:
// exact softmax attention over the selected key blocks) on the dequantised
// operands Q = sq * q8, K = sk * k8, V = sv * v8, where every block of
// tokens carries one power-of-two scale.  The scales enter the matrix cores
// as E8M0 block scales of v_mfma_scale_f32_32x32x64_f8f6f4, so the scores come
// out dequantised with no extra VALU work.
//
// One wavefront per 64-row query tile, one wave per SIMD, no LDS: K and V
// arrive in the matrix cores' operand order (written so by the tile-layout
// quantisation), so each key tile is two sets of eight 16-byte loads per
// lane, every load instruction reading 1 KB contiguous, issued one tile
// ahead.  A key tile is used by exactly one wave, so nothing would be shared
// through LDS.  Per 64-key tile:
//   S^T (64 keys x 64 queries) = K . Q^T    8 x v_mfma_scale_..._32x32x64 (scales sk, sq),
//                                           one half of the queries at a time
//   P = 2^(x - m) * 2^(8 - kLazy) as e4m3 codes built directly: the code of
//       2^y, linear in the mantissa between integer y, is 8 (y + 7), so each
//       score costs one FMA and one v_cvt_pk_u8_f32 that rounds it to a byte
//       and packs it (exact at integer exponents, linear in between)
//   O^T (128 x 64)        += V^T . P^T        8 x v_mfma_scale_..._32x32x64 (scales sv, 2^(kLazy-8))
//   row sums of P          += 1^T . P^T        2 more MFMAs against an all-ones channel
// so the normaliser is the sum of exactly the rounded probabilities the PV
// product uses, accumulated (and rescaled) by the matrix cores.  The next
// tile's first score products are issued before the current tile's PV
// products, so the softmax of one runs while the matrix cores work on the
// other.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kRowBytes = kHeadDim;             // 128 B per e4m3 row
constexpr int kOpTileBytes = kTile * kRowBytes; // 8 KB: one 64-key tile in operand order
constexpr float kLazy = 2.f;  // log2 headroom of P above the reference before a shift
constexpr int kMaxShift = 100;  // largest shift of P's frame (keeps fp32 sums finite)
constexpr float kLog2PScale = 6.f;               // log2 of 2^(8 - kLazy): P in (0, 256] before e4m3
constexpr int kPScaleInvE8m0 = 127 - 6;          // E8M0 code of 2^-(8 - kLazy)
constexpr int kOneE8m0 = 127;                    // E8M0 code of 1
constexpr int kFp8One = 0x38383838;              // four e4m3 ones

typedef __attribute__((__vector_size__(2 * sizeof(int)))) int i32x2;
typedef const __attribute__((address_space(4))) int32_t* list_ptr;
typedef const __attribute__((address_space(4))) float* scale_ptr;

struct Params {
  const uint8_t* q;
  const uint8_t* k;
  const uint8_t* v;
  const float* sq;
  const float* sk;
  const float* sv;
  uint16_t* o;
  float* lse;
  Strides os;
  const int32_t* idx;
  const int32_t* cnt;
  const int32_t* order;
  int kmax, H, N, block, nb, ntiles;
  float scale_log2;
  Shape cs;  // causal window (causal_chunk 0: none)
};

// Scalar load of element `i` (non-negative) of a uniform array: the byte
// offset stays a 32-bit SGPR operand of s_load (one shift) instead of a
// 64-bit address computed per load.
template <typename T>
__device__ __forceinline__ T sld(const __attribute__((address_space(4))) T* base, uint32_t i) {
  return *reinterpret_cast<const __attribute__((address_space(4))) T*>(
      reinterpret_cast<const __attribute__((address_space(4))) char*>(base) + i * (uint32_t)sizeof(T));
}

__device__ __forceinline__ int tile_start(list_ptr list, int n, int spb, int block, int nb,
                                          int N) {
  const int e = n >> (spb - 1);  // spb (sub-tiles per block) is 1 or 2
  const int j = sld(list, (uint32_t)e);
  if (j < 0 || j >= nb) return -1;
  const int st = j * block + (n - (e << (spb - 1))) * kTile;
  return st < N ? st : -1;
}

__device__ __forceinline__ int next_tile(list_ptr list, int n, int total, int spb, int block,
                                         int nb, int N, int* start) {
  for (; n < total; ++n) {
    const int st = tile_start(list, n, spb, block, nb, N);
    if (st >= 0) {
      *start = st;
      return n;
    }
  }
  return total;
}

// E8M0 code of a power-of-two fp32 scale (its biased exponent).
__device__ __forceinline__ int e8m0(float s) { return (int)((__float_as_uint(s) >> 23) & 0xffu); }


__global__ __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(1, 1))) void fwd_fp8_kernel(
    Params p) {
  const int item = p.order ? p.order[blockIdx.x] : (int)blockIdx.x;
  const int bh = item / p.ntiles;
  const int qt = item - bh * p.ntiles;
  const int b = bh / p.H, h = bh - b * p.H;
  const int q0 = qt * kTile;
  const int iblk = q0 / p.block;
  const int spb = p.block / kTile;
  // List and scales are read-only here: reading them through the constant
  // address space makes the uniform reads scalar loads.
  const list_ptr list = (list_ptr)(p.idx + ((int64_t)bh * p.nb + iblk) * p.kmax);
  const int c = min(max(p.cnt[(int64_t)bh * p.nb + iblk], 0), p.kmax);
  const int total = c * spb;
  const int lane = threadIdx.x & (kWave - 1);
  const int g = lane >> 5, l32 = lane & 31;

  // Allowed keys [key_lo, key_hi) of this lane's queries (one per half of
  // the tile); a tile needs the per-score mask unless it lies inside every
  // row's range: [lo of the tile's last row, hi of its first).
  int key_lo[2], key_hi[2];
#pragma unroll
  for (int qh = 0; qh < 2; ++qh) {
    const int qtok = min(q0 + 32 * qh + l32, p.N - 1);
    key_lo[qh] = causal_lo(p.cs, qtok);
    key_hi[qh] = causal_hi(p.cs, qtok);
  }
  const int tile_lo = causal_lo(p.cs, min(q0 + kTile - 1, p.N - 1));
  const int tile_hi = causal_hi(p.cs, q0);

  const int64_t qhead = (int64_t)bh * p.N * kRowBytes;
  const auto qr = make_rsrc(p.q + qhead, (uint32_t)p.N * kRowBytes);
  const int64_t ophead = (int64_t)bh * p.ntiles * kOpTileBytes;
  const uint32_t opbytes = (uint32_t)p.ntiles * kOpTileBytes;
  const auto kr = make_rsrc(p.k + ophead, opbytes);
  const auto vr = make_rsrc(p.v + ophead, opbytes);
  const scale_ptr skh = (scale_ptr)(p.sk + (int64_t)bh * p.nb);
  const scale_ptr svh = (scale_ptr)(p.sv + (int64_t)bh * p.nb);
  const int sq_code = e8m0(((scale_ptr)p.sq)[(int64_t)bh * p.nb + iblk]);

  // Q fragments (B operand of K . Q^T): query q0 + 32 qh + l32, bytes
  // 64 ks + 32 g .. +31 of its row (rows past N read as zeros).
  i32x8 qf[2][2];
#pragma unroll
  for (int qh = 0; qh < 2; ++qh)
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const uint32_t off = (uint32_t)(q0 + 32 * qh + l32) * kRowBytes + 64 * ks + 32 * g;
      const u32x4 lo = buf_ld16(qr, off), hi = buf_ld16(qr, off + 16);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        qf[qh][ks][x] = (int)lo[x];
        qf[qh][ks][4 + x] = (int)hi[x];
      }
    }

  // Operand-order tile loads (t: 64-key tile of the head): K fragment
  // (rt, ks) = chunks 2 (2 rt + ks) and 2 (2 rt + ks) + 1, V^T fragment dt =
  // chunks 2 dt and 2 dt + 1, each chunk 1 KB (16 bytes per lane).
  auto load_k = [&](i32x8 (&kf)[2][2], int t) __attribute__((always_inline)) {
    const uint32_t base = (uint32_t)__builtin_amdgcn_readfirstlane(t) * kOpTileBytes;
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const u32x4 lo = buf_ld16(kr, 16 * lane + 2048 * f, base);
      const u32x4 hi = buf_ld16(kr, 16 * lane + 2048 * f + 1024, base);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        kf[f >> 1][f & 1][x] = (int)lo[x];
        kf[f >> 1][f & 1][4 + x] = (int)hi[x];
      }
    }
  };
  auto load_v = [&](i32x8 (&vf)[4], int t) __attribute__((always_inline)) {
    const uint32_t base = (uint32_t)__builtin_amdgcn_readfirstlane(t) * kOpTileBytes;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const u32x4 lo = buf_ld16(vr, 16 * lane + 2048 * dt, base);
      const u32x4 hi = buf_ld16(vr, 16 * lane + 2048 * dt + 1024, base);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        vf[dt][x] = (int)lo[x];
        vf[dt][4 + x] = (int)hi[x];
      }
    }
  };

  // O^T per query half, and the row sums of both halves in registers 0 and
  // 1 of lanes 0..31 (rows 0 and 1 of one 32x32 product)
  f32x16 acc[2][4], accl;
  // all-ones row qh of the row-sum A operand: lanes holding row qh
  i32x8 ones[2];
#pragma unroll
  for (int qh = 0; qh < 2; ++qh)
#pragma unroll
    for (int x = 0; x < 8; ++x) ones[qh][x] = l32 == qh ? kFp8One : 0;
  // Reference max per query (log2 units), fixed for the whole row once set:
  // a tile whose max lies above it by more than kLazy computes its P against
  // ref + e (e a whole number) and enters the products with the extra scale
  // 2^e through the per-lane E8M0 scale of the P operand, so no vector
  // instruction ever rescales the accumulators.  A shift beyond kMaxShift
  // (fp32 headroom) restarts the row from its first tile with the new max.
  float mref[2] = {-INFINITY, -INFINITY};
  const float cexp8 = p.scale_log2 * 8.f;  // 8 tau log2(e)
  bool restart = false;

  // Keys outside the causal window or past N get a score of -inf; a tile
  // needs the per-score test unless it lies inside every row's range: [lo
  // of the tile's last row, hi of its first).  The test runs between the
  // pipeline's blocks, only for such tiles.
  auto needs_mask = [&](int start) __attribute__((always_inline)) {
    return start + kTile > tile_hi || start < tile_lo;
  };
  auto apply_mask = [&](f32x16 (&s)[2], int start, int qh) __attribute__((always_inline)) {
    int st = __builtin_amdgcn_readfirstlane(start);
    asm volatile("" : "+s"(st));
    const int hi = key_hi[qh] - st - 4 * g, lo = key_lo[qh] - st - 4 * g;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int off = 32 * rt + 8 * (r >> 2) + (r & 3);  // key - start - 4g
        if (off >= hi || off < lo) s[rt][r] = -INFINITY;
      }
  };

  // S^T of one tile for query half qh: lane holds keys 32 rt + 8 (r / 4) +
  // 4 g + r % 4 of query 32 qh + l32
  auto scores = [&](const i32x8 (&kf)[2][2], int sk_code, int qh, f32x16 (&s)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      s[rt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf[rt][0], qf[qh][0], (f32x16){}, 0,
                                                              0, 0, sk_code, 0, sq_code);
      s[rt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf[rt][1], qf[qh][1], s[rt], 0, 0,
                                                              0, sk_code, 0, sq_code);
    }
  };

  // Softmax numerators of one tile for query half qh: P^T as the B operand,
  // slot 16 rt + r <- s[rt][r], values 2^(x - ref - e) * 2^(8 - kLazy) in
  // e4m3; bscale = E8M0 code of 2^(e - (8 - kLazy)).  Branch-free (a shift
  // beyond kMaxShift only raises `restart`).
  auto softmax = [&](const f32x16 (&s)[2], int qh, i32x8& pk, int& bscale) __attribute__((always_inline)) {
    float mx = s[0][0];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[rt][r]);
    mx = pair_max32(mx) * p.scale_log2;  // the tile's max for this query (both lanes)
    const float ref = mref[qh] == -INFINITY ? mx : mref[qh];  // first tile with an allowed key
    const float over = mx - ref - kLazy;  // NaN (both -inf) and -inf give e = 0
    int e = over > 0.f ? (int)__builtin_ceilf(over) : 0;
    const bool far = e > kMaxShift;
    restart |= __any(far);
    mref[qh] = far ? mx : ref;
    e = far ? 0 : e;
    bscale = kPScaleInvE8m0 + e;
    // P * 2^6 = 2^y with y = tau*log2(e)*s - ref - e + 6 <= kLazy + 6 = 8, as
    // the e4m3 code 8 (y + 7) rounded to an integer: exponent field
    // floor(y) + 7, mantissa the first 3 bits of the fraction, i.e. 2^y exact
    // at integer y and linear in between (at most 6.2% above 2^y, the same
    // relative excess for a given fraction), at most 120 (2^8; 127 would be
    // NaN).  v_cvt_pk_u8_f32 rounds to nearest, ties to even, and clamps to
    // [0, 255] (NaN to 0), measured by an in-bounds probe: y < -7 and masked scores
    // (-inf) give code 0, P = 0; codes 1..7 (y in [-7, -6)) read as e4m3
    // subnormals, at most 2^-15 of the tile's largest P.
    const float mloc = mref[qh] == -INFINITY ? 0.f : mref[qh] + (float)e;
    const float kexp8 = (kLog2PScale + 7.f - mloc) * 8.f;  // 8 (6 + 7 - m): the e4m3 bias
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 16; r += 4) {
        uint32_t w = 0u;
#pragma unroll
        for (int u = 0; u < 4; ++u)
          w = __builtin_amdgcn_cvt_pk_u8_f32(fmaf(s[rt][r + u], cexp8, kexp8), u, w);
        pk[4 * rt + r / 4] = (int)w;
      }
  };

  // O^T += V^T . P^T and row sums += 1^T . P^T for one tile
  auto pv = [&](const i32x8 (&vf)[4], const i32x8 (&pk)[2], int sv_code, const int (&bs)[2]) __attribute__((always_inline)) {
#pragma unroll
    for (int qh = 0; qh < 2; ++qh) {
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
        acc[qh][dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            vf[dt], pk[qh], acc[qh][dt], 0, 0, 0, sv_code, 0, bs[qh]);
      accl = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ones[qh], pk[qh], accl, 0, 0, 0,
                                                             kOneE8m0, 0, bs[qh]);
    }
  };

  auto block_of = [&](int n) __attribute__((always_inline)) { return n < total ? sld(list, (uint32_t)(n >> (spb - 1))) : 0; };
#pragma unroll
  for (int qh = 0; qh < 2; ++qh)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[qh][dt][r] = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) accl[r] = 0.f;

  // Software pipeline over the list.  Tile 0 is the current tile n, tile 1
  // the next, tile 2 the one after (n == total: none; a missing tile is
  // replaced by tile 0, whose products are then discarded).  On entry to a
  // step: P(n, half 0) in pk[0], S(n, half 1) in sa, V(n) in vf, K(n+1) in kf.
  // A step computes, in blocks whose matrix and vector work interleave,
  //   [1] S(n+1, half 0)           with  softmax(n, half 1)
  //   [2] S(n+1, half 1), then K(n+2) starts to load into kf
  //   [3] PV(n)                    with  softmax(n+1, half 0)
  // and V(n+1) loads once PV(n) has been issued.  P(n+1, half 0) overwrites
  // P(n, half 0) after the products that read it have been issued.
  int st0 = p.N, st1 = p.N;
  const int n_first = next_tile(list, 0, total, spb, p.block, p.nb, p.N, &st0);
  const int st_first = st0;
  if (n_first < total) {
    i32x8 kf[2][2], vf[4], pk[2];
    int bs[2];
    f32x16 sa[2], sb[2];
    int n0 = 0, n1 = 0, j0 = 0, j1 = 0;
    // read one step ahead (scalar loads): the list entry after tile 1, the
    // K scale of tile 1 and the V scale of tile 0
    int raw = 0;
    float skf = 1.f, svf = 1.f;
    auto prefetch = [&]() __attribute__((always_inline)) {
      raw = sld(list, (uint32_t)min((n1 + 1) >> (spb - 1), p.kmax - 1));
      skf = sld(skh, j1);
      svf = sld(svh, j0);
    };
    auto prologue = [&]() __attribute__((always_inline)) {
      n0 = n_first;
      st0 = st_first;
      n1 = next_tile(list, n0 + 1, total, spb, p.block, p.nb, p.N, &st1);
      j0 = block_of(n0);
      j1 = block_of(n1);
      load_k(kf, st0 >> 6);
      load_v(vf, st0 >> 6);
      const int sk0 = e8m0(sld(skh, j0));
      scores(kf, sk0, 0, sb);
      scores(kf, sk0, 1, sa);
      load_k(kf, (n1 < total ? st1 : st0) >> 6);
      if (needs_mask(st0)) {
        apply_mask(sb, st0, 0);
        apply_mask(sa, st0, 1);
      }
      softmax(sb, 0, pk[0], bs[0]);
      prefetch();
    };
    for (;;) {
    prologue();
    for (;;) {
      const bool has1 = n1 < total;
      const int sv0 = e8m0(svf), sk1 = e8m0(skf);
      // tile 2: the prefetched entry decodes it unless it is invalid (then
      // the list is scanned)
      int n2 = total, st2 = p.N, j2 = 0;
      if (has1 && n1 + 1 < total) {
        const int j = __builtin_amdgcn_readfirstlane(raw);
        const int s0 = j * p.block + ((n1 + 1) & (spb - 1)) * kTile;
        if (j >= 0 && j < p.nb && s0 < p.N) {
          n2 = n1 + 1;
          st2 = s0;
          j2 = j;
        } else {
          n2 = next_tile(list, n1 + 2, total, spb, p.block, p.nb, p.N, &st2);
          j2 = block_of(n2);
        }
      }
      const int st1x = has1 ? st1 : st0;
      const bool m1 = needs_mask(st1x);
      // [1]
      scores(kf, sk1, 0, sb);
      softmax(sa, 1, pk[1], bs[1]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
        __builtin_amdgcn_sched_group_barrier(0x002, 28, 0);  // then vector work
      }
      __builtin_amdgcn_sched_barrier(0);
      // [2]
      scores(kf, sk1, 1, sa);
      load_k(kf, (n2 < total ? st2 : st0) >> 6);
      if (m1) {
        apply_mask(sb, st1x, 0);
        apply_mask(sa, st1x, 1);
      }
      // [3]
      pv(vf, pk, sv0, bs);
      softmax(sb, 0, pk[0], bs[0]);
#pragma unroll
      for (int i = 0; i < 10; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 12, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      load_v(vf, st1x >> 6);
      if (restart) break;
      if (!has1) break;
      n0 = n1;
      st0 = st1;
      j0 = j1;
      n1 = n2;
      st1 = st2;
      j1 = j2;
      prefetch();
    }
    if (!restart) break;
    // a shift beyond kMaxShift: start over from the first tile with the
    // raised reference (products with zero operands clear the sums)
    restart = false;
    const i32x8 z = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int qh = 0; qh < 2; ++qh)
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
        acc[qh][dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            z, z, (f32x16){}, 0, 0, 0, kOneE8m0, 0, kOneE8m0);
    accl = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(z, z, (f32x16){}, 0, 0, 0,
                                                           kOneE8m0, 0, kOneE8m0);
    }
  }

  // ---- normalise, store ---------------------------------------------------
#pragma unroll
  for (int qh = 0; qh < 2; ++qh) {
    // the row sum of query 32 qh + l32 sits in register qh of lane l32
    const float l = __shfl(accl[qh], l32, kWave);
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const int row = q0 + 32 * qh + l32;
    if (row < p.N) {
      uint16_t* op = p.o + b * p.os.b + h * p.os.h + (int64_t)row * p.os.n;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          u32x2 w;
          w[0] = pack_bf16x2(acc[qh][dt][4 * j] * inv, acc[qh][dt][4 * j + 1] * inv);
          w[1] = pack_bf16x2(acc[qh][dt][4 * j + 2] * inv, acc[qh][dt][4 * j + 3] * inv);
          *reinterpret_cast<u32x2*>(op + dt * 32 + 8 * j + 4 * g) = w;
        }
      }
      if (p.lse && g == 0)
        p.lse[(int64_t)bh * p.N + row] =
            l > 0.f ? (mref[qh] + __builtin_amdgcn_logf(l)) * 0.69314718055994531f : -INFINITY;
    }
  }
}

}  // namespace

hipError_t launch_fwd_fp8(const Shape& s, const FwdArgs& a, hipStream_t stream) {
  Params p;
  p.q = static_cast<const uint8_t*>(a.q);
  p.k = static_cast<const uint8_t*>(a.k);
  p.v = static_cast<const uint8_t*>(a.v);
  p.sq = a.sq;
  p.sk = a.sk;
  p.sv = a.sv;
  p.o = static_cast<uint16_t*>(a.o);
  p.lse = a.lse;
  p.os = a.os;
  p.idx = a.idx;
  p.cnt = a.cnt;
  p.order = a.order;
  p.kmax = a.kmax;
  p.H = s.H;
  p.N = s.N;
  p.block = s.block;
  p.nb = s.nb;
  p.ntiles = (s.N + kTile - 1) / kTile;
  p.scale_log2 = a.softmax_scale * 1.4426950408889634f;
  p.cs = s;
  fwd_fp8_kernel<<<s.B * s.H * p.ntiles, kWave, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace sa

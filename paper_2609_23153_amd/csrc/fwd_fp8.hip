// Fused block-sparse attention forward on fp8 (OCP e4m3) operands, gfx950.
//
// The same result as the bf16 forward (paper §2 Eq. comp-sparse, §4.1:
// exact softmax attention over the selected key blocks) on the dequantised
// operands Q = sq * q8, K = sk * k8, V = sv * v8, where every block of
// tokens carries one power-of-two scale.  The scales enter the matrix cores
// as E8M0 block scales of v_mfma_scale_f32_32x32x64_f8f6f4, so the scores come
// out dequantised with no extra VALU work.
//
// One workgroup = 4 wavefronts = one 64-row query tile; two workgroups share
// a CU.  A 32x32x64 fp8 MFMA contracts 64 keys, so each wave takes a whole
// 64-key tile: waves 0/1 own query rows 0-31 / 32-63 of the first tile of
// each pair of tiles in the list, waves 2/3 of the second.  Per wave and tile:
//   S^T (64 keys x 32 queries) = K . Q^T       4 x v_mfma_scale_..._32x32x64 (scales sk, sq)
//   P = 2^(x - m) * 2^(8 - kLazy) rounded to e4m3 with v_cvt_pk_fp8_f32, the
//       power of two built in integer arithmetic (one FMA and one conversion
//       per score: exact at integer exponents, linear in between)
//   O^T (128 x 32)        += V^T . P^T        4 x v_mfma_scale_..._32x32x64 (scales sv, 2^(kLazy-8))
//   row sums of P          += 1^T . P^T        1 more MFMA against an all-ones channel
// so the normaliser is the sum of exactly the rounded probabilities the PV
// product uses, accumulated (and rescaled) by the matrix cores.
// Copies: pairs of K and V tiles go global -> LDS with buffer_load ... lds
// issued from inline asm.  K pairs are double- and V pairs triple-buffered
// (80 KB of LDS): each step reads its K fragments, releases the K buffer at
// one barrier and refills it with the pair two steps ahead; the V buffer the
// previous step read is refilled at the start of the step.  The V^T operand
// is read from the row-major V tile with ds_read_b64_tr_b8.  The two
// tile-parity waves of a row-half merge their softmax states at the end.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kThreads = 256;
constexpr int kRowBytes = kHeadDim;             // 128 B per e4m3 row
constexpr int kTileBytes = kTile * kRowBytes;   // 8 KB per K or V tile
constexpr int kPairBytes = 2 * kTileBytes;      // one pair of tiles
constexpr float kLazy = 2.f;  // log2 headroom before the accumulator is rescaled
constexpr float kPScale = 64.f;                  // 2^(8 - kLazy): P in (0, 256] before e4m3
constexpr float kLog2PScale = 6.f;               // log2(kPScale)
constexpr int kPScaleInvE8m0 = 127 - 6;          // E8M0 code of 2^-(8 - kLazy)
constexpr int kOneE8m0 = 127;                    // E8M0 code of 1
constexpr int kFp8One = 0x38383838;              // four e4m3 ones

// 16-byte-chunk swizzles of 128-byte rows (row = row within the tile):
// conflict-free for the K A-operand reads (16 rows, one chunk per pass) and
// the V transpose reads (rows k0 + {0..3, 8..11}, two chunks per pass).
__device__ __forceinline__ int swz_k(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }
__device__ __forceinline__ int swz_v(int row, int chunk) {
  return chunk ^ ((((row >> 1) & 1) << 1) | (((row >> 3) & 1) << 2));
}

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

// v_cvt_u32_f32: truncation to an unsigned integer with the hardware's
// saturation (negative values and NaN give 0, values >= 2^32 give
// 0xffffffff), written as asm because C++ leaves negative inputs undefined.
__device__ __forceinline__ uint32_t cvt_u32_sat(float x) {
  uint32_t u;
  asm("v_cvt_u32_f32 %0, %1" : "=v"(u) : "v"(x));
  return u;
}

// E8M0 code of a power-of-two fp32 scale (its biased exponent).
__device__ __forceinline__ int e8m0(float s) { return (int)((__float_as_uint(s) >> 23) & 0xffu); }

// Global byte offset of the logical chunk that the swizzle stores at LDS slot
// `slot` of tile row `row`.
__device__ __forceinline__ uint32_t dma_offset(int row, int slot, bool is_v) {
  const int chunk = is_v ? swz_v(row, slot) : swz_k(row, slot);
  return (uint32_t)row * kRowBytes + (uint32_t)chunk * 16u;
}

// s_waitcnt with the other counters at their maxima (no wait on them).
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }
__device__ __forceinline__ void wait_vm8() { __builtin_amdgcn_s_waitcnt(0x0F78); }
__device__ __forceinline__ void wait_vm16() { __builtin_amdgcn_s_waitcnt(0x4F70); }
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

__global__ __launch_bounds__(kThreads, 2) void fwd_fp8_kernel(Params p) {
  // Distinct LDS objects per buffer keep every access at a constant base.
  __shared__ __attribute__((aligned(1024))) uint8_t kp0[kPairBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t kp1[kPairBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vp0[kPairBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vp1[kPairBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vp2[kPairBytes];

  const int item = p.order ? p.order[blockIdx.x] : (int)blockIdx.x;
  const int bh = item / p.ntiles;
  const int qt = item - bh * p.ntiles;
  const int b = bh / p.H, h = bh - b * p.H;
  const int q0 = qt * kTile;
  const int iblk = q0 / p.block;
  const int spb = p.block / kTile;
  // List and scales are read-only here: reading them through the constant
  // address space makes the uniform reads scalar loads, which vmcnt does not
  // count.
  const list_ptr list = (list_ptr)(p.idx + ((int64_t)bh * p.nb + iblk) * p.kmax);
  const int c = min(max(p.cnt[(int64_t)bh * p.nb + iblk], 0), p.kmax);
  const int total = c * spb;

  // the wave index is uniform across a wave: read it into a scalar register
  // so that everything derived from it (the tile a wave computes, its
  // scales, the mask test) stays scalar
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int rh = wave & 1, par = wave >> 1;  // row half, tile parity
  const int g = lane >> 5, l32 = lane & 31;

  // Allowed keys [key_lo, key_hi) of this lane's query (the causal window,
  // and the sequence end); a tile needs the per-score mask unless it lies
  // inside every row's range: [lo of the tile's last row, hi of its first).
  const int qtok = min(q0 + rh * 32 + l32, p.N - 1);
  const int key_lo = causal_lo(p.cs, qtok), key_hi = causal_hi(p.cs, qtok);
  const int tile_lo = causal_lo(p.cs, min(q0 + kTile - 1, p.N - 1));
  const int tile_hi = causal_hi(p.cs, q0);

  const int64_t head = (int64_t)bh * p.N * kRowBytes;
  const uint32_t bytes = (uint32_t)p.N * kRowBytes;
  const auto kr = make_rsrc(p.k + head, bytes);
  const auto vr = make_rsrc(p.v + head, bytes);
  const scale_ptr skh = (scale_ptr)(p.sk + (int64_t)bh * p.nb);
  const scale_ptr svh = (scale_ptr)(p.sv + (int64_t)bh * p.nb);
  const int sq_code = e8m0(((scale_ptr)p.sq)[(int64_t)bh * p.nb + iblk]);

  // Copies of a pair into [tile A | tile B]: each wave moves rows 16w .. 16w+15
  // of each tile (two 1 KB copies of 8 rows), lane l writing LDS slot l%8 of
  // row l/8 of those 8 rows.
  uint32_t koff[2], voff[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = 16 * wave + 8 * i + (lane >> 3);
    koff[i] = dma_offset(row, lane & 7, false);
    voff[i] = dma_offset(row, lane & 7, true);
  }
  const int wv = __builtin_amdgcn_readfirstlane(wave);
  auto dma_pair = [&](uint8_t* dst, __amdgpu_buffer_rsrc_t r, const uint32_t (&off)[2], int a0,
                      int b0) {
    // the wave's row offset passes through an opaque move, so the compiler
    // adds the constant buffer offsets per copy instead of holding every
    // (buffer, copy) address live across the loop
    uint32_t wrow;
    asm volatile("s_mov_b32 %0, %1" : "=s"(wrow) : "s"((uint32_t)(16 * wv) * kRowBytes));
    const uint32_t base = lds_addr(dst) + wrow;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 2; ++i)
        dma16(base + t * kTileBytes + 8 * i * kRowBytes, r, off[i],
              (uint32_t)(t ? b0 : a0) * kRowBytes);
  };

  // Pair cursor: pairs P0 (being computed), P1 and P2 as start rows (ta*,
  // tb*; N when missing: such tiles read zeros and all their keys are
  // masked, and the loop ends when P0 has no first tile) and key blocks (ja*,
  // jb*); nb2 is the list position of the last tile taken.  The list entries
  // after P2 and the scales of P1 are read one step ahead.
  auto block_of = [&](int n) { return n < total ? sld(list, (uint32_t)(n >> (spb - 1))) : 0; };
  int ta0 = p.N, tb0 = p.N, ta1 = p.N, tb1 = p.N, ta2 = p.N, tb2 = p.N;
  const int na0 = next_tile(list, 0, total, spb, p.block, p.nb, p.N, &ta0);
  const int nb0 = next_tile(list, na0 + 1, total, spb, p.block, p.nb, p.N, &tb0);
  const int na1 = next_tile(list, nb0 + 1, total, spb, p.block, p.nb, p.N, &ta1);
  const int nb1 = next_tile(list, na1 + 1, total, spb, p.block, p.nb, p.N, &tb1);
  const int na2 = next_tile(list, nb1 + 1, total, spb, p.block, p.nb, p.N, &ta2);
  int nb2 = next_tile(list, na2 + 1, total, spb, p.block, p.nb, p.N, &tb2);
  int ja1 = block_of(na1), jb1 = block_of(nb1);
  int ja2 = block_of(na2), jb2 = block_of(nb2);
  // scale codes of the current pair: (K, V) for tiles A and B
  const int ja0 = block_of(na0), jb0 = block_of(nb0);
  int sk_a = e8m0(sld(skh, ja0)), sv_a = e8m0(sld(svh, ja0)), sk_b = e8m0(sld(skh, jb0)),
      sv_b = e8m0(sld(svh, jb0));

  // Prologue: the Q tile is staged through vp2 (K swizzle) while the K and V
  // pairs P0 and P1 are issued; step 0 refills vp2 with V(P2) once every wave
  // holds its Q fragment.  Every step issues the same number of copies, so
  // the vmcnt arithmetic below is uniform.
  {
    const auto qr = make_rsrc(p.q + head, bytes);
    const uint32_t base = lds_addr(vp2) + (uint32_t)(16 * wv) * kRowBytes;
#pragma unroll
    for (int i = 0; i < 2; ++i) dma16(base + 8 * i * kRowBytes, qr, koff[i], (uint32_t)q0 * kRowBytes);
  }
  dma_pair(kp0, kr, koff, ta0, tb0);
  dma_pair(vp0, vr, voff, ta0, tb0);
  dma_pair(vp1, vr, voff, ta1, tb1);
  dma_pair(kp1, kr, koff, ta1, tb1);
  wait_vm16();  // this wave's rows of Q have landed
  barrier_keep_loads();

  // Q fragment (B operand of K.Q^T): query row 32*rh + l32, bytes
  // 64*ks + 32*g .. +31 of the row.
  i32x8 qf[2];
  {
    const int row = rh * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c0 = 4 * ks + 2 * g;
      const u32x4 lo = *reinterpret_cast<const u32x4*>(vp2 + row * kRowBytes + swz_k(row, c0) * 16);
      const u32x4 hi = *reinterpret_cast<const u32x4*>(vp2 + row * kRowBytes + swz_k(row, c0 + 1) * 16);
#pragma unroll
      for (int x = 0; x < 4; ++x) {
        qf[ks][x] = (int)lo[x];
        qf[ks][4 + x] = (int)hi[x];
      }
    }
  }
  wait_lgkm0();
  barrier_keep_loads();  // vp2 (Q) is free for V(P2)

  f32x16 acc[4], accl;  // O^T, and the row sums in register 0 of lanes 0..31
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[dt][r] = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) accl[r] = 0.f;
  // all-ones channel 0 of the row-sum A operand: lanes holding channel 0
  i32x8 ones;
#pragma unroll
  for (int x = 0; x < 8; ++x) ones[x] = l32 == 0 ? kFp8One : 0;
  float m2 = -INFINITY;

  // V^T transpose read: lane 16G + 2e + h supplies the 8 bytes of key
  // 16a + 8(e>>2) + 4(G>>1) + (e&3) at channels 32*dt + 16(G&1) + 8h .. +7;
  // lane l then holds channel 32*dt + (l&31) of slots 8a .. 8a+7.
  const int G = lane >> 4, e8 = (lane >> 1) & 7, h8 = lane & 1;
  const int vrow0 = 8 * (e8 >> 2) + 4 * (G >> 1) + (e8 & 3);  // + 16a

  wait_vm8();  // K(P0), V(P0) landed (V(P1), K(P1) may still fly)
  barrier_keep_loads();

  // Next valid tile at or after index `ahead` whose raw list entry `pre`
  // was prefetched: the common case decodes it directly, an invalid entry
  // falls back to a scan of the list.
  auto advance = [&](int ahead, int pre, int* st, int* jout) {
    *st = p.N;
    *jout = 0;
    if (ahead >= total) return total;
    const int j = __builtin_amdgcn_readfirstlane(pre);
    const int s0 = j * p.block + (ahead & (spb - 1)) * kTile;
    if (j >= 0 && j < p.nb && s0 < p.N) {
      *st = s0;
      *jout = j;
      return ahead;
    }
    const int m = next_tile(list, ahead + 1, total, spb, p.block, p.nb, p.N, st);
    *jout = block_of(m);
    return m;
  };

  // One pair: compute from K pair buffer `kc` and V pair buffer `vc`; `vn`
  // (read by the previous step) receives V(P2) at once and `kc` receives
  // K(P2) after the barrier that follows the K fragment reads.
  auto step = [&](uint8_t* kc, const uint8_t* vc, uint8_t* vn) {
    dma_pair(vn, vr, voff, ta2, tb2);
    const uint8_t* kt = kc + par * kTileBytes;
    i32x8 kf[2][2];  // [row tile][k-step]
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      const int row = rt * 32 + l32;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int c0 = 4 * ks + 2 * g;
        const u32x4 lo = *reinterpret_cast<const u32x4*>(kt + row * kRowBytes + swz_k(row, c0) * 16);
        const u32x4 hi =
            *reinterpret_cast<const u32x4*>(kt + row * kRowBytes + swz_k(row, c0 + 1) * 16);
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          kf[rt][ks][x] = (int)lo[x];
          kf[rt][ks][4 + x] = (int)hi[x];
        }
      }
    }
    // one step ahead: scales of P1, list entries after P2
    const float fka = sld(skh, ja1), fva = sld(svh, ja1), fkb = sld(skh, jb1), fvb = sld(svh, jb1);
    const int pre1 = sld(list, (uint32_t)min((nb2 + 1) >> (spb - 1), p.kmax - 1));
    const int pre2 = sld(list, (uint32_t)min((nb2 + 2) >> (spb - 1), p.kmax - 1));
    wait_lgkm0();
    barrier_keep_loads();  // every wave holds its K fragments: kc is free
    dma_pair(kc, kr, koff, ta2, tb2);

    const uint8_t* vt = vc + par * kTileBytes;
    i32x8 vf[4];
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int lc = 2 * dt + (G & 1);  // logical 16-B chunk of channels 32dt + 16(G&1)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int row = vrow0 + 16 * a;
        const i32x2 t = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
            (__attribute__((address_space(3))) i32x2*)(vt + row * kRowBytes +
                                                       swz_v(row, lc) * 16 + h8 * 8));
        vf[dt][2 * a] = t[0];
        vf[dt][2 * a + 1] = t[1];
      }
    }

    const int start = par ? tb0 : ta0;
    const int sk_code = par ? sk_b : sk_a;
    const int sv_code = par ? sv_b : sv_a;

    // ---- S^T = K . Q^T (two 32-key row tiles) -----------------------------
    f32x16 s[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[rt][r] = 0.f;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
        s[rt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf[rt][ks], qf[ks], s[rt], 0, 0,
                                                                 0, sk_code, 0, sq_code);
    }
    // lane holds keys 32*rt + 8*(r>>2) + 4*g + (r&3) of query l32
    if (start + kTile > tile_hi || start < tile_lo) {
      // (the opaque move keeps the per-key arithmetic inside the branch)
      int st = __builtin_amdgcn_readfirstlane(start);
      asm volatile("" : "+s"(st));
      const int hi = key_hi - st - 4 * g, lo = key_lo - st - 4 * g;
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int off = 32 * rt + 8 * (r >> 2) + (r & 3);  // key - start - 4g
          if (off >= hi || off < lo) s[rt][r] = -INFINITY;
        }
    }

    // ---- online softmax --------------------------------------------------
    float mx = s[0][0];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[rt][r]);
    mx *= p.scale_log2;
    if (__any(mx > m2 + kLazy)) {  // wave-uniform: raise the reference max
      const float mnew = fmaxf(m2, pair_max32(mx));
      const float alpha = __builtin_amdgcn_exp2f(m2 - (mnew == -INFINITY ? 0.f : mnew));
      accl[0] *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[dt][r] *= alpha;
      m2 = mnew;
    }
    const float msafe = m2 == -INFINITY ? 0.f : m2;
    // P^T as B operand: slot 16*rt + r <- s[rt][r]; values 2^(x - m) * 2^(8 - kLazy)
    // rounded to e4m3
    i32x8 pk;
    // P * 2^6 = 2^y with y = tau*log2(e)*s - m + 6, as the fp32 whose bit
    // pattern is (y + 127) * 2^23 truncated to an integer: exact at integer
    // y and linear in the mantissa between them (at most 6.2% above 2^y, the
    // same relative excess for a given fractional part of y).  One FMA and
    // one conversion per score instead of an FMA and a transcendental; the
    // e4m3 rounding that follows keeps 3 mantissa bits anyway.  Negative
    // patterns (y < -127, and masked scores) convert to 0, i.e. P = 0.
    const float cexp = p.scale_log2 * 8388608.f;                    // tau log2(e) 2^23
    const float kexp = (kLog2PScale + 127.f - msafe) * 8388608.f;  // (6 + 127 - m) 2^23
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
      for (int r = 0; r < 16; r += 4) {
        float x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
          x[u] = __uint_as_float(cvt_u32_sat(fmaf(s[rt][r + u], cexp, kexp)));
        int w = __builtin_amdgcn_cvt_pk_fp8_f32(x[0], x[1], 0, false);
        w = __builtin_amdgcn_cvt_pk_fp8_f32(x[2], x[3], w, true);
        pk[4 * rt + r / 4] = w;
      }
    }

    // ---- O^T += V^T . P^T, row sums += 1^T . P^T ----------------------------
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
      acc[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vf[dt], pk, acc[dt], 0, 0, 0,
                                                                sv_code, 0, kPScaleInvE8m0);
    accl = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(ones, pk, accl, 0, 0, 0, kOneE8m0, 0,
                                                           kPScaleInvE8m0);

    // advance the cursor
    ta0 = ta1;
    tb0 = tb1;
    ta1 = ta2;
    tb1 = tb2;
    ja1 = ja2;
    jb1 = jb2;
    sk_a = e8m0(fka);
    sv_a = e8m0(fva);
    sk_b = e8m0(fkb);
    sv_b = e8m0(fvb);
    const int prev = nb2;
    const int n2 = advance(prev + 1, pre1, &ta2, &ja2);
    if (n2 == prev + 1) {
      nb2 = advance(n2 + 1, pre2, &tb2, &jb2);
    } else {
      nb2 = next_tile(list, n2 + 1, total, spb, p.block, p.nb, p.N, &tb2);
      jb2 = block_of(nb2);
    }
    // keep the whole pair's work ahead of the wait
    __builtin_amdgcn_sched_barrier(0);
    wait_vm8();  // K(P1), V(P1) landed; V(P2), K(P2) may fly
    barrier_keep_loads();  // also: every wave is done reading vc
  };
  // step n reads K pair buffer n%2 and V pair buffer n%3, refills V (n+2)%3
  while (ta0 < p.N) {
    step(kp0, vp0, vp2);
    if (ta0 >= p.N) break;
    step(kp1, vp1, vp0);
    if (ta0 >= p.N) break;
    step(kp0, vp2, vp1);
    if (ta0 >= p.N) break;
    step(kp1, vp0, vp2);
    if (ta0 >= p.N) break;
    step(kp0, vp1, vp0);
    if (ta0 >= p.N) break;
    step(kp1, vp2, vp1);
  }
  wait_vm0();
  __syncthreads();

  // ---- merge the two tile-parity waves, normalise, store -----------------
  // the row sum of query l32 sits in register 0 of lane l32
  float lsum = __shfl(accl[0], l32, kWave);
  float* mrg = reinterpret_cast<float*>(rh ? vp0 : kp0);  // 66 x 64 floats per row-half
  if (par == 1) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mrg[(dt * 16 + r) * kWave + lane] = acc[dt][r];
    mrg[64 * kWave + lane] = m2;
    mrg[65 * kWave + lane] = lsum;
  }
  __syncthreads();
  if (par == 0) {
    const float m_o = mrg[64 * kWave + lane];
    const float l_o = mrg[65 * kWave + lane];
    const float mm = fmaxf(m2, m_o);
    const float ms = mm == -INFINITY ? 0.f : mm;
    const float a0 = __builtin_amdgcn_exp2f(m2 - ms);
    const float a1 = __builtin_amdgcn_exp2f(m_o - ms);
    const float l = lsum * a0 + l_o * a1;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const float c0 = a0 * inv, c1 = a1 * inv;
    const int row = q0 + rh * 32 + l32;
    if (row < p.N) {
      uint16_t* op = p.o + b * p.os.b + h * p.os.h + (int64_t)row * p.os.n;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          float x[4];
#pragma unroll
          for (int r = 0; r < 4; ++r)
            x[r] = acc[dt][4 * j + r] * c0 + mrg[(dt * 16 + 4 * j + r) * kWave + lane] * c1;
          u32x2 w;
          w[0] = pack_bf16x2(x[0], x[1]);
          w[1] = pack_bf16x2(x[2], x[3]);
          *reinterpret_cast<u32x2*>(op + dt * 32 + 8 * j + 4 * g) = w;
        }
      }
      if (p.lse && g == 0)
        p.lse[(int64_t)bh * p.N + row] =
            l > 0.f ? (mm + __builtin_amdgcn_logf(l)) * 0.69314718055994531f : -INFINITY;
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
  fwd_fp8_kernel<<<s.B * s.H * p.ntiles, kThreads, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace sa

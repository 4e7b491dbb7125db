// Fused block-sparse attention forward on fp8 (OCP e4m3) operands, gfx950.
//
// The same result as the bf16 forward (paper §2 Eq. comp-sparse, §4.1:
// exact softmax attention over the selected key blocks) on the dequantised
// operands Q = sq * q8, K = sk * k8, V = sv * v8, where every block of
// tokens carries one power-of-two scale.  The scales enter the matrix cores
// as E8M0 block scales of v_mfma_scale_f32_32x32x64_f8f6f4, so the scores come
// out dequantised with no extra VALU work.
//
// One workgroup = 4 wavefronts = one 64-row query tile.  A 32x32x64 fp8 MFMA
// contracts 64 keys, so each wave takes a whole 64-key tile: waves 0/1 own
// query rows 0-31 / 32-63 of the even tiles of the list, waves 2/3 of the
// odd tiles; every step moves two tiles (K and V, 32 KB) global -> LDS with
// buffer_load ... lds, double-buffered.  Per wave and tile:
//   S^T (64 keys x 32 queries) = K . Q^T       4 x v_mfma_scale_..._32x32x64 (scales sk, sq)
//   P = 2^(x - m) * 2^(8 - kLazy) rounded to e4m3 with v_cvt_pk_fp8_f32
//   O^T (128 x 32)        += V^T . P^T        4 x v_mfma_scale_..._32x32x64 (scales sv, 2^(kLazy-8))
// The V^T operand is read from the row-major V tile with ds_read_b64_tr_b8.
// The two tile-parity waves of a row-half merge their softmax states at the end.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kThreads = 256;
constexpr int kRowBytes = kHeadDim;             // 128 B per e4m3 row
constexpr int kTileBytes = kTile * kRowBytes;   // 8 KB per K or V tile
constexpr int kBufBytes = 4 * kTileBytes;       // two tiles x (K, V) = 32 KB
constexpr float kLazy = 2.f;  // log2 headroom before the accumulator is rescaled
constexpr float kPScale = 64.f;                  // 2^(8 - kLazy): P in (0, 256] before e4m3
constexpr int kPScaleInvE8m0 = 127 - 6;          // E8M0 code of 2^-(8 - kLazy)

// 16-byte-chunk swizzles of 128-byte rows (row = row within the tile):
// conflict-free for the K A-operand reads (16 rows, one chunk per pass) and
// the V transpose reads (rows k0 + {0..3, 8..11}, two chunks per pass).
__device__ __forceinline__ int swz_k(int row, int chunk) { return chunk ^ ((row >> 1) & 7); }
__device__ __forceinline__ int swz_v(int row, int chunk) {
  return chunk ^ ((((row >> 1) & 1) << 1) | (((row >> 3) & 1) << 2));
}

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((__vector_size__(2 * sizeof(int)))) int i32x2;

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
};

__device__ __forceinline__ int tile_start(const int32_t* list, int n, int spb, int block,
                                          int nb, int N) {
  const int e = n / spb;
  const int j = list[e];
  if (j < 0 || j >= nb) return -1;
  const int st = j * block + (n - e * spb) * kTile;
  return st < N ? st : -1;
}

__device__ __forceinline__ int next_tile(const int32_t* list, int n, int total, int spb,
                                         int block, int nb, int N, int* start) {
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

// Global byte offset of the logical chunk that the swizzle stores at LDS slot
// `slot` of tile row `row`.
__device__ __forceinline__ uint32_t dma_offset(int row, int slot, bool is_v) {
  const int chunk = is_v ? swz_v(row, slot) : swz_k(row, slot);
  return (uint32_t)row * kRowBytes + (uint32_t)chunk * 16u;
}

__device__ __forceinline__ void wait_dma() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__global__ __launch_bounds__(kThreads, 2) void fwd_fp8_kernel(Params p) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds0[kBufBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t lds1[kBufBytes];

  const int item = p.order ? p.order[blockIdx.x] : (int)blockIdx.x;
  const int bh = item / p.ntiles;
  const int qt = item - bh * p.ntiles;
  const int b = bh / p.H, h = bh - b * p.H;
  const int q0 = qt * kTile;
  const int iblk = q0 / p.block;
  const int spb = p.block / kTile;
  const int32_t* list = p.idx + ((int64_t)bh * p.nb + iblk) * p.kmax;
  const int c = min(max(p.cnt[(int64_t)bh * p.nb + iblk], 0), p.kmax);
  const int total = c * spb;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rh = wave & 1, par = wave >> 1;  // row half, tile parity
  const int g = lane >> 5, l32 = lane & 31;

  const int64_t head = (int64_t)bh * p.N * kRowBytes;
  const uint32_t bytes = (uint32_t)p.N * kRowBytes;
  const auto kr = make_rsrc(p.k + head, bytes);
  const auto vr = make_rsrc(p.v + head, bytes);
  const float* skh = p.sk + (int64_t)bh * p.nb;
  const float* svh = p.sv + (int64_t)bh * p.nb;
  const int sq_code = e8m0(p.sq[(int64_t)bh * p.nb + iblk]);

  // Copies: a step moves two tiles A and B into [K_A | K_B | V_A | V_B]; each
  // wave copies rows 16w .. 16w+15 of each (two 1 KB instructions of 8 rows),
  // lane l writing LDS slot l%8 of row l/8 of those 8 rows.
  uint32_t koff[2], voff[2];
  {
    const int w = threadIdx.x >> 6;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int row = 16 * w + 8 * i + (lane >> 3);
      koff[i] = dma_offset(row, lane & 7, false);
      voff[i] = dma_offset(row, lane & 7, true);
    }
  }
  auto dma = [&](uint8_t* dst, int a0, int b0) {
    const int w = threadIdx.x >> 6;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const uint32_t soff = (uint32_t)(t ? b0 : a0) * kRowBytes;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int r0 = 16 * w + 8 * i;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            kr, (lds_void*)(dst + t * kTileBytes + r0 * kRowBytes), 16, koff[i], soff, 0, 0);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            vr, (lds_void*)(dst + (2 + t) * kTileBytes + r0 * kRowBytes), 16, voff[i], soff, 0,
            0);
      }
    }
  };

  // Tile cursor: the current pair (na0, ta) / (nb0, tb) with key blocks
  // ja / jb, and the next pair (na1, ua) / (nb1, ub).  Missing tiles start at
  // N: they read zeros and all their keys are masked.  The list entries of
  // the pair after next and the scales of the next pair are read one step
  // ahead, alongside that step's copies, so no step waits on them.
  auto block_of = [&](int n) { return n < total ? list[n / spb] : 0; };
  int ta = p.N, tb = p.N, ua = p.N, ub = p.N;
  int na0 = next_tile(list, 0, total, spb, p.block, p.nb, p.N, &ta);
  int nb0 = next_tile(list, na0 + 1, total, spb, p.block, p.nb, p.N, &tb);
  int na1 = next_tile(list, nb0 + 1, total, spb, p.block, p.nb, p.N, &ua);
  int nb1 = next_tile(list, na1 + 1, total, spb, p.block, p.nb, p.N, &ub);
  int ja = block_of(na0), jb = block_of(nb0), ka = block_of(na1), kb = block_of(nb1);
  if (na0 < total) dma(lds0, ta, tb);
  // scale codes of the current pair: (K, V) for tiles A and B
  int sk_a = e8m0(skh[ja]), sv_a = e8m0(svh[ja]), sk_b = e8m0(skh[jb]), sv_b = e8m0(svh[jb]);

  // Q fragment (B operand of K.Q^T): query row l32 of this row-half, bytes
  // 64*ks + 32*g .. +31 of the row.
  i32x8 qf[2];
  {
    const auto qr = make_rsrc(p.q + head, bytes);
    const uint32_t off = (uint32_t)(q0 + rh * 32 + l32) * kRowBytes + g * 32;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const u32x4 lo = buf_ld16(qr, off + ks * 64), hi = buf_ld16(qr, off + ks * 64 + 16);
      for (int x = 0; x < 4; ++x) {
        qf[ks][x] = (int)lo[x];
        qf[ks][4 + x] = (int)hi[x];
      }
    }
  }

  f32x16 acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[dt][r] = 0.f;
  float m2 = -INFINITY;
  float lsum = 0.f;

  // V^T transpose read: lane 16G + 2e + h supplies the 8 bytes of key
  // 16a + 8(e>>2) + 4(G>>1) + (e&3) at channels 32*dt + 16(G&1) + 8h .. +7;
  // lane l then holds channel 32*dt + (l&31) of slots 8a .. 8a+7.
  const int G = lane >> 4, e8 = (lane >> 1) & 7, h8 = lane & 1;
  const int vrow0 = 8 * (e8 >> 2) + 4 * (G >> 1) + (e8 & 3);  // + 16a

  wait_dma();
  __syncthreads();

  // Next valid tile at or after index `ahead` whose raw list entry `pre`
  // was prefetched: the common case decodes it directly, an invalid entry
  // falls back to a scan of the list.
  auto advance = [&](int ahead, int pre, int* st, int* jout) {
    *st = p.N;
    *jout = 0;
    if (ahead >= total) return total;
    const int j = __builtin_amdgcn_readfirstlane(pre);
    const int s0 = j * p.block + (ahead % spb) * kTile;
    if (j >= 0 && j < p.nb && s0 < p.N) {
      *st = s0;
      *jout = j;
      return ahead;
    }
    const int m = next_tile(list, ahead + 1, total, spb, p.block, p.nb, p.N, st);
    *jout = block_of(m);
    return m;
  };

  auto step = [&](const uint8_t* cur, uint8_t* nxt) {
    dma(nxt, ua, ub);
    // one step ahead: scales of the next pair, list entries after it
    const float fka = skh[ka], fva = svh[ka], fkb = skh[kb], fvb = svh[kb];
    const int pre1 = list[min((nb1 + 1) / spb, p.kmax - 1)];
    const int pre2 = list[min((nb1 + 2) / spb, p.kmax - 1)];

    const int start = par ? tb : ta;
    const uint8_t* kt = cur + par * kTileBytes;
    const uint8_t* vt = cur + (2 + par) * kTileBytes;
    const int sk_code = par ? sk_b : sk_a;
    const int sv_code = par ? sv_b : sv_a;

    // ---- S^T = K . Q^T (two 32-key row tiles) -----------------------------
    f32x16 s[2];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[rt][r] = 0.f;
      const int row = rt * 32 + l32;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int c0 = 4 * ks + 2 * g;
        const u32x4 lo = *reinterpret_cast<const u32x4*>(kt + row * kRowBytes + swz_k(row, c0) * 16);
        const u32x4 hi =
            *reinterpret_cast<const u32x4*>(kt + row * kRowBytes + swz_k(row, c0 + 1) * 16);
        i32x8 kf;
        for (int x = 0; x < 4; ++x) {
          kf[x] = (int)lo[x];
          kf[4 + x] = (int)hi[x];
        }
        s[rt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kf, qf[ks], s[rt], 0, 0, 0,
                                                                 sk_code, 0, sq_code);
      }
    }
    // lane holds keys 32*rt + 8*(r>>2) + 4*g + (r&3) of query l32
    if (start + kTile > p.N) {
#pragma unroll
      for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = start + 32 * rt + 8 * (r >> 2) + 4 * g + (r & 3);
          if (key >= p.N) s[rt][r] = -INFINITY;
        }
    }

    // ---- online softmax --------------------------------------------------
    float mx = s[0][0];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[rt][r]);
    mx *= p.scale_log2;
    if (__any(mx > m2 + kLazy)) {
      const float mnew = fmaxf(m2, pair_max32(mx));
      const float alpha = __builtin_amdgcn_exp2f(m2 - (mnew == -INFINITY ? 0.f : mnew));
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[dt][r] *= alpha;
      m2 = mnew;
    }
    const float msafe = m2 == -INFINITY ? 0.f : m2;
    // P^T as B operand: slot 16*rt + r <- s[rt][r]; values 2^(x - m) * 2^(8 - kLazy)
    // rounded to e4m3, the exact pre-rounding values summed into lsum.
    i32x8 pk;
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
#pragma unroll
      for (int r = 0; r < 16; r += 4) {
        float x[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          x[u] = __builtin_amdgcn_exp2f(fmaf(s[rt][r + u], p.scale_log2, -msafe));
          lsum += x[u];
        }
        int w = __builtin_amdgcn_cvt_pk_fp8_f32(x[0] * kPScale, x[1] * kPScale, 0, false);
        w = __builtin_amdgcn_cvt_pk_fp8_f32(x[2] * kPScale, x[3] * kPScale, w, true);
        pk[4 * rt + r / 4] = w;
      }
    }

    // ---- O^T += V^T . P^T ------------------------------------------------
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int lc = 2 * dt + (G & 1);  // logical 16-B chunk of channels 32dt + 16(G&1)
      i32x8 vf;
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const int row = vrow0 + 16 * a;
        const i32x2 t = __builtin_amdgcn_ds_read_tr8_b64_v2i32(
            (__attribute__((address_space(3))) i32x2*)(vt + row * kRowBytes +
                                                       swz_v(row, lc) * 16 + h8 * 8));
        vf[2 * a] = t[0];
        vf[2 * a + 1] = t[1];
      }
      acc[dt] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vf, pk, acc[dt], 0, 0, 0, sv_code,
                                                                0, kPScaleInvE8m0);
    }

    wait_dma();
    __syncthreads();
    na0 = na1;
    nb0 = nb1;
    ta = ua;
    tb = ub;
    sk_a = e8m0(fka);
    sv_a = e8m0(fva);
    sk_b = e8m0(fkb);
    sv_b = e8m0(fvb);
    const int prev = nb1;
    na1 = advance(prev + 1, pre1, &ua, &ka);
    if (na1 == prev + 1) {
      nb1 = advance(na1 + 1, pre2, &ub, &kb);
    } else {
      nb1 = next_tile(list, na1 + 1, total, spb, p.block, p.nb, p.N, &ub);
      kb = block_of(nb1);
    }
  };
  while (na0 < total) {
    step(lds0, lds1);
    if (na0 >= total) break;
    step(lds1, lds0);
  }

  // ---- merge the two tile-parity waves, normalise, store -----------------
  lsum += __shfl_xor(lsum, 32, kWave);
  float* mrg = reinterpret_cast<float*>(rh ? lds1 : lds0);  // 66 x 64 floats per row-half
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
  fwd_fp8_kernel<<<s.B * s.H * p.ntiles, kThreads, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace sa

// Fused block-sparse attention forward, bf16 operands, for gfx950.
//
// Computes the sparse branch A_M of compensated sparse attention (paper §2
// Eq. comp-sparse, §4.1): exact softmax attention of each 64-row query tile
// over the union of the key blocks its query block selected.
//
// One workgroup = 4 wavefronts = one 64-row query tile; two workgroups share
// a CU.  Every selected key block is walked as 64-key tiles:
//  * K and V tiles go straight from L2 into LDS with buffer_load ... lds (no
//    staging registers, no VALU), rows past the sequence end reading zero
//    through the buffer range check.  Both are stored row-major with a
//    16-byte-chunk XOR swizzle chosen on the global side.
//  * K is double- and V triple-buffered (80 KB of LDS per workgroup).  Step n
//    first refills the V buffer step n-1 read with V(n+2), then reads its K
//    fragments into registers; after one barrier the K buffer is free and
//    receives K(n+2), and the V^T fragments of step n are read while the S
//    products run.  A K tile has about a step and a half, a V tile two, to
//    arrive: enough bytes in flight to cover L2 latency under load.
//  * Wave w owns query rows 32*(w&1)..+31 and keys 32*(w>>1)..+31 of a tile:
//      S^T (32 keys x 32 queries) = K_half . Q_half^T   8 x v_mfma_f32_32x32x16_bf16
//      O^T (128 x 32)          += V_half^T . P^T       8 x v_mfma_f32_32x32x16_bf16
//    Computing S transposed leaves all 16 scores of a lane in one query
//    column: row statistics are per-lane scalars and the probabilities are
//    already in the B-operand layout of the PV product.  The V^T A-operand is
//    read from the row-major V tile with ds_read_b64_tr_b16.
//  * Online softmax in fp32 registers with exp2 (tau*log2(e) folded into one
//    FMA) and a lazily raised reference max: the common tile costs one FMA
//    and one exp2 per score, a bf16 pack per pair and a v_dot2 per pair for
//    the row sum; the max is only taken on the tiles that raise it.
// The two key-half waves of a row-half keep separate softmax states that are
// merged through LDS at the end.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kThreads = 256;
constexpr int kRowBytes = kHeadDim * 2;            // 256 B per bf16 row
constexpr int kTileBytes = kTile * kRowBytes;      // 16 KB per K or V tile

// A tile's probabilities are taken against the running reference max as it
// stands; only when a lane's tile sum of them exceeds this bound (or is not
// finite) is the max raised and the tile recomputed, so every probability
// stays <= kSumCap.
constexpr float kSumCap = 4096.f;

// 16-byte-chunk swizzles (row = row within the tile): conflict-free for the
// K A-operand reads (32 rows, one chunk) and the V transpose reads (4 rows x
// 4 chunks per half-wave).
__device__ __forceinline__ int swz_k(int row, int chunk) { return chunk ^ (row & 15); }
__device__ __forceinline__ int swz_v(int row, int chunk) { return chunk ^ ((row & 3) << 2); }

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;

struct Params {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  Strides qs, ks, vs, os;
  const int32_t* idx;
  const int32_t* cnt;
  const int32_t* order;
  int kmax, H, N, block, nb, ntiles;  // ntiles = ceil(N / 64) query tiles per head
  float scale_log2;                   // tau * log2(e)
  Shape cs;                           // causal window (causal_chunk 0: none)
};

// Start row of the n-th 64-key tile of a query block's list, or -1 when the
// list entry is out of range or the sub-tile lies past the sequence end.
typedef const __attribute__((address_space(4))) int32_t* list_ptr;

__device__ __forceinline__ int tile_start(list_ptr list, int n, int sh, int block, int nb,
                                          int N) {
  const int e = n >> sh;
  const int j = list[e];
  if (j < 0 || j >= nb) return -1;
  const int st = j * block + (n - (e << sh)) * kTile;
  return st < N ? st : -1;
}

__device__ __forceinline__ int next_tile(list_ptr list, int n, int total, int sh, int block,
                                         int nb, int N, int* start) {
  for (; n < total; ++n) {
    const int st = tile_start(list, n, sh, block, nb, N);
    if (st >= 0) {
      *start = st;
      return n;
    }
  }
  return total;
}

// Per-lane global byte offsets (loop invariant) of the 16-byte chunks this
// lane moves into LDS: wave w, instruction i covers tile rows 16w+4i .. +3,
// lane l writes LDS chunk slot l%16 of row 16w+4i+l/16 and so fetches the
// logical chunk that the swizzle places there.
struct DmaOffsets {
  uint32_t k[4];
  uint32_t v[4];
};

__device__ __forceinline__ DmaOffsets dma_offsets(uint32_t kst, uint32_t vst) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  DmaOffsets o;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 16 * w + 4 * i + (l >> 4);
    o.k[i] = (uint32_t)row * kst + (uint32_t)swz_k(row, l & 15) * 16u;
    o.v[i] = (uint32_t)row * vst + (uint32_t)swz_v(row, l & 15) * 16u;
  }
  return o;
}

// Issue the global -> LDS copies of one K or V tile (4 instructions per
// wave, each 4 rows); completion is tracked by vmcnt, which the caller waits.
__device__ __forceinline__ void dma_tile(uint8_t* dst, __amdgpu_buffer_rsrc_t r,
                                         const uint32_t (&off)[4], uint32_t soff) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t base = lds_addr(dst) + (uint32_t)(16 * w) * kRowBytes;
#pragma unroll
  for (int i = 0; i < 4; ++i) dma16(base + 4 * i * kRowBytes, r, off[i], soff);
}

// s_waitcnt with the other counters at their maxima (no wait on them).
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }
__device__ __forceinline__ void wait_vm8() { __builtin_amdgcn_s_waitcnt(0x0F78); }
__device__ __forceinline__ void wait_vm16() { __builtin_amdgcn_s_waitcnt(0x4F70); }
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Probabilities 2^(s*c - m) of a lane's 16 scores packed to bf16 as the PV
// B operand (k-step cs in pk[cs]), and their sum over those bf16 values
// (v_dot2 against (1, 1)), so numerator and normaliser see the same numbers.
__device__ __forceinline__ float tile_probs(const f32x16& s, float c, float m, bf16x8 (&pk)[2]) {
  const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
  float ts = 0.f;
#pragma unroll
  for (int cs = 0; cs < 2; ++cs) {
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float a = __builtin_amdgcn_exp2f(fmaf(s[8 * cs + 2 * e], c, -m));
      const float b = __builtin_amdgcn_exp2f(fmaf(s[8 * cs + 2 * e + 1], c, -m));
      const bf16x2 t = {(__bf16)a, (__bf16)b};
      w[e] = __builtin_bit_cast(uint32_t, t);
      ts = __builtin_amdgcn_fdot2_f32_bf16(t, one, ts, false);
    }
    pk[cs] = __builtin_bit_cast(bf16x8, w);
  }
  return ts;
}

__global__ __launch_bounds__(kThreads, 2) void fwd_bf16_kernel(Params p) {
  // Distinct LDS objects per buffer (rather than one array indexed by a
  // buffer number) keep every access at a constant base.
  __shared__ __attribute__((aligned(1024))) uint8_t kb0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t kb1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vb0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vb1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vb2[kTileBytes];

  const int item = p.order ? p.order[blockIdx.x] : (int)blockIdx.x;
  const int bh = item / p.ntiles;
  const int qt = item - bh * p.ntiles;
  const int b = bh / p.H, h = bh - b * p.H;
  const int q0 = qt * kTile;
  const int iblk = q0 / p.block;
  const int spb = p.block / kTile;
  const int sh = spb == 2 ? 1 : 0;  // log2(spb): blocks are 64 or 128 tokens
  const int c = min(max(p.cnt[(int64_t)bh * p.nb + iblk], 0), p.kmax);
  const int total = c * spb;
  // The list is read-only here: reading it through the constant address space
  // makes the uniform reads scalar loads (s_load), which vmcnt does not count.
  const list_ptr list = (list_ptr)(p.idx + ((int64_t)bh * p.nb + iblk) * p.kmax);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rh = wave & 1, kh = wave >> 1;
  const int g = lane >> 5, l32 = lane & 31;

  // Allowed keys [key_lo, key_hi) of this lane's query (the causal window,
  // and the sequence end); a tile needs the per-score mask unless it lies
  // inside every row's range: [lo of the tile's last row, hi of its first).
  const int qtok = min(q0 + rh * 32 + l32, p.N - 1);
  const int key_lo = causal_lo(p.cs, qtok), key_hi = causal_hi(p.cs, qtok);
  const int tile_lo = causal_lo(p.cs, min(q0 + kTile - 1, p.N - 1));
  const int tile_hi = causal_hi(p.cs, q0);

  // Per-head buffer resources covering rows [0, N): rows past N read zero.
  const uint32_t kst = (uint32_t)p.ks.n * 2, vst = (uint32_t)p.vs.n * 2, qst = (uint32_t)p.qs.n * 2;
  const auto kr = make_rsrc(p.k + b * p.ks.b + h * p.ks.h, (uint32_t)(p.N - 1) * kst + 256u);
  const auto vr = make_rsrc(p.v + b * p.vs.b + h * p.vs.h, (uint32_t)(p.N - 1) * vst + 256u);
  const DmaOffsets dofs = dma_offsets(kst, vst);

  // Tile cursor: n / s0 = tile being computed, n1, n2 / s1, s2 = the next
  // two valid tiles (total / N when there are none).  The list entry after
  // n2 is read one step ahead.
  int s0 = p.N, s1 = p.N, s2 = p.N;
  int n = next_tile(list, 0, total, sh, p.block, p.nb, p.N, &s0);
  int n1 = next_tile(list, n + 1, total, sh, p.block, p.nb, p.N, &s1);
  int n2 = next_tile(list, n1 + 1, total, sh, p.block, p.nb, p.N, &s2);

  // Prologue.  The Q tile is staged through vb2 (same swizzle as K) while
  // K(0), V(0), V(1), K(1) are issued; step 0 refills vb2 with V(2) once every
  // wave holds its Q fragment.  Past the end of the list the starts equal N
  // and the copies read zeros without touching memory, so every step issues
  // the same number of copies and the vmcnt arithmetic below is uniform.
  {
    const auto qr = make_rsrc(p.q + b * p.qs.b + h * p.qs.h, (uint32_t)(p.N - 1) * qst + 256u);
    const DmaOffsets qofs = dma_offsets(qst, qst);
    dma_tile(vb2, qr, qofs.k, (uint32_t)q0 * qst);
  }
  dma_tile(kb0, kr, dofs.k, (uint32_t)s0 * kst);
  dma_tile(vb0, vr, dofs.v, (uint32_t)s0 * vst);
  dma_tile(vb1, vr, dofs.v, (uint32_t)s1 * vst);
  dma_tile(kb1, kr, dofs.k, (uint32_t)s1 * kst);
  wait_vm16();  // this wave's rows of Q have landed
  barrier_keep_loads();

  // LDS read addresses (bytes, relative to a buffer):
  //  Q B-operand / K A-operand: row rh*32 + l32 / kh*32 + l32, logical chunk
  //  2*ks + g.
  //  V^T A-operand (transpose read): lane 16G + 4e + q supplies the 8-byte
  //  chunk of key kh*32 + 16*cs + 8*hf + 4*(G>>1) + e at channels
  //  32*dt + 16*(G&1) + 4*q .. +3; lane l then receives channel 32*dt + (l&31)
  //  of keys kh*32 + 16*cs + 8*hf + 4*g + {0..3}.
  const int krow = kh * 32 + l32;
  // K read of k-step ks at (kx ^ 32*ks): the chunk swizzle (2*ks + g) ^ (krow & 15)
  // splits into ks ^ (krow >> 1 & 7) (bits 5..7 of the offset) and g ^ (krow & 1)
  const uint32_t kx = (uint32_t)krow * kRowBytes + (uint32_t)(((krow >> 1) & 7) << 5) +
                      (uint32_t)((g ^ (krow & 1)) << 4);
  const int G = lane >> 4, e4 = (lane >> 2) & 3, q4 = lane & 3;
  const int vrow0 = kh * 32 + 4 * (G >> 1) + e4;  // + 16*cs + 8*hf (keeps row & 3)

  // Q fragment (B operand of K.Q^T): query row l32 of this row-half,
  // channels 16*ks + 8*g .. +7.
  bf16x8 qf[8];
  {
    const int qrow = rh * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      qf[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(vb2 + qrow * kRowBytes +
                                                         swz_k(qrow, 2 * ks + g) * 16));
  }
  wait_lgkm0();
  barrier_keep_loads();  // vb2 (Q) is free for V(2)

  f32x16 acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[dt][r] = 0.f;
  // Reference max (log2 domain, tau*log2(e)*logit) of this lane's query: the
  // accumulator holds sum 2^(x - m2) v.  It starts at -inf, so the first tile
  // always sets it, and is raised only when a tile's probabilities would
  // exceed kSumCap.  Lanes l and l^32 share one query and one m2.
  float m2 = -INFINITY;
  float lsum = 0.f;  // partial sum of the bf16 probabilities over this lane's keys

  wait_vm8();  // K(0), V(0) landed (V(1), K(1) may still fly)
  barrier_keep_loads();

  // One 64-key tile, computed from K buffer `kc` and V buffer `vc`.  Step n
  // first refills `vn` (the buffer step n-1 read) with V(n+2); after its K
  // fragments are in registers and one barrier, `kc` receives K(n+2).  The
  // V^T fragments are read after that barrier and land during the S MFMAs.
  auto step = [&](uint8_t* kc, const uint8_t* vc, uint8_t* vn) {
    dma_tile(vn, vr, dofs.v, (uint32_t)s2 * vst);
    // derive the 8 K read offsets here each step (one XOR each) rather than
    // keeping 8 loop-invariant registers live across the loop
    uint32_t kxs = kx;
    asm volatile("" : "+v"(kxs));
    bf16x8 kf[8];
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      kf[ks] = as_bf16x8(*reinterpret_cast<const u32x4*>(kc + (kxs ^ (uint32_t)(ks << 5))));
    // list entry of the tile after n2 (a scalar load, waited below)
    const int ahead = n2 + 1;
    const int pre = list[min(ahead >> sh, p.kmax - 1)];
    wait_lgkm0();
    barrier_keep_loads();  // every wave holds its K fragments: kc is free
    dma_tile(kc, kr, dofs.k, (uint32_t)s2 * kst);
    u32x4 vf[8];  // V^T fragments, [2*dt + cs]
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      const int lc = 4 * dt + 2 * (G & 1) + (q4 >> 1);  // logical 16-B chunk
      const int half = (q4 & 1) * 8;
#pragma unroll
      for (int cs = 0; cs < 2; ++cs)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int row = vrow0 + 16 * cs + 8 * hf;
          const i16x4 t = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) i16x4*)(vc + row * kRowBytes +
                                                         swz_v(row, lc) * 16 + half));
          const u32x2 tw = __builtin_bit_cast(u32x2, t);
          vf[2 * dt + cs][2 * hf] = tw[0];
          vf[2 * dt + cs][2 * hf + 1] = tw[1];
        }
    }

    // ---- S^T = K_half . Q^T ------------------------------------------------
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks], qf[ks], s, 0, 0, 0);
    // lane holds keys kh*32 + 8*(r>>2) + 4*g + (r&3) of query l32
    if (s0 + kTile > tile_hi || s0 < tile_lo) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = s0 + kh * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
        if (key >= key_hi || key < key_lo) s[r] = -INFINITY;
      }
    }

    // ---- online softmax --------------------------------------------------
    // P^T as B operand: k-step cs uses registers 8cs .. 8cs+7 (keys
    // 16cs + 4g + {0..3} and 16cs + 8 + 4g + {0..3} of the half).  The tile
    // sum is taken over the bf16 values the PV product uses (v_dot2 against
    // (1, 1)), so numerator and normaliser see the same probabilities.
    bf16x8 pk[2];
    // with m2 = -inf every probability is +inf or NaN, so the first tile
    // always takes the branch
    float ts = tile_probs(s, p.scale_log2, m2, pk);
    if (__any(!(ts <= kSumCap))) {  // wave-uniform: raise the reference max
      float mx = s[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[r]);
      mx *= p.scale_log2;
      const float mnew = fmaxf(m2, pair_max32(mx));
      const float msafe = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = __builtin_amdgcn_exp2f(m2 - msafe);
      lsum *= alpha;
#pragma unroll
      for (int dt = 0; dt < 4; ++dt)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[dt][r] *= alpha;
      m2 = mnew;
      ts = tile_probs(s, p.scale_log2, msafe, pk);
    }
    lsum += ts;

    // ---- O^T += V_half^T . P^T -------------------------------------------
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int cs = 0; cs < 2; ++cs)
        acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vf[2 * dt + cs]), pk[cs],
                                                          acc[dt], 0, 0, 0);

    // advance the cursor
    n = n1;
    n1 = n2;
    s0 = s1;
    s1 = s2;
    s2 = p.N;
    n2 = total;
    if (ahead < total) {
      const int j = __builtin_amdgcn_readfirstlane(pre);
      const int st = j * p.block + (ahead & (spb - 1)) * kTile;
      if (j >= 0 && j < p.nb && st < p.N) {
        n2 = ahead;
        s2 = st;
      } else {
        n2 = next_tile(list, ahead + 1, total, sh, p.block, p.nb, p.N, &s2);
      }
    }
    // keep the whole tile's work ahead of the wait
    __builtin_amdgcn_sched_barrier(0);
    wait_vm8();  // K(n+1), V(n+1) landed; V(n+2), K(n+2) may fly
    barrier_keep_loads();  // also: every wave is done reading vc
  };
  // step n reads K[n%2] and V[n%3] and refills V[(n+2)%3] and K[n%2]
  while (n < total) {
    step(kb0, vb0, vb2);
    if (n >= total) break;
    step(kb1, vb1, vb0);
    if (n >= total) break;
    step(kb0, vb2, vb1);
    if (n >= total) break;
    step(kb1, vb0, vb2);
    if (n >= total) break;
    step(kb0, vb1, vb0);
    if (n >= total) break;
    step(kb1, vb2, vb1);
  }
  wait_vm0();
  __syncthreads();

  // ---- merge the two key halves, normalise, store ------------------------
  lsum += __shfl_xor(lsum, 32, kWave);
  // per row-half: 64 x 64 accumulator floats in kb0 / kb1 (16 KB each), the
  // max and sum (2 x 64 floats) in vb0
  float* mrg = reinterpret_cast<float*>(rh ? kb1 : kb0);
  float* mls = reinterpret_cast<float*>(vb0) + rh * 2 * kWave;
  if (kh == 1) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mrg[(dt * 16 + r) * kWave + lane] = acc[dt][r];
    mls[lane] = m2;
    mls[kWave + lane] = lsum;
  }
  __syncthreads();
  if (kh == 0) {
    const float m_o = mls[lane];
    const float l_o = mls[kWave + lane];
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

hipError_t launch_fwd_bf16(const Shape& s, const FwdArgs& a, hipStream_t stream) {
  Params p;
  p.q = static_cast<const uint16_t*>(a.q);
  p.k = static_cast<const uint16_t*>(a.k);
  p.v = static_cast<const uint16_t*>(a.v);
  p.o = static_cast<uint16_t*>(a.o);
  p.lse = a.lse;
  p.qs = a.qs;
  p.ks = a.ks;
  p.vs = a.vs;
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
  const int grid = s.B * s.H * p.ntiles;
  fwd_bf16_kernel<<<grid, kThreads, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace sa

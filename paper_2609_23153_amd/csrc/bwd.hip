// Backward pass of the block-sparse attention forward (the sparse branch of
// paper §2 Eq. comp-sparse; its gradients serve the training of the sparse
// model, §2 "Training sparse attention" and the Stage-1 warm-up of §4.4),
// bf16 operands, gfx950.  Per query block i with key set U_i (its selected
// blocks), with P = softmax(tau Q_i K_U^T) rebuilt from the forward's LSE:
//   dV_U += P^T dO_i,  dP = dO_i V_U^T,  dS = P o (dP - D_i),
//   dQ_i = tau dS K_U,  dK_U += tau dS^T Q_i,  D_i = rowsum(dO_i o O_i).
//
// Kernels:
//  * bwd_dot_kernel: D = rowsum(dO o O) in fp32, one 16-lane group per token;
//  * bwd_bits_clear / bwd_bits_set: the transposed selection as a bitmap,
//    bit i of row j set when query block i selected key block j (atomic OR,
//    order independent, so the result is deterministic);
//  * bwd_dq_kernel: one workgroup per 64-row query tile walks its list like
//    the forward (wave (rh, kh): query rows 32 rh.., keys 32 kh.. of a tile):
//      S^T = K Q^T, dP^T = V dO^T (8 + 8 MFMAs), P and dS per lane,
//      dQ^T += K^T dS^T (8 MFMAs, K^T by transposed LDS reads);
//    the two key halves are summed at the end;
//  * bwd_dkdv_kernel: one workgroup per 64-key tile walks the query blocks
//    that selected its key block (set bits of its bitmap row, ascending) in
//    two phases per query tile: S^T and dP^T per (key half, query half),
//    P and dS through LDS, then dV^T += dO^T P and dK^T += Q^T dS per (key
//    half, channel half) over the whole tile.
// Every product is a bf16 32x32x16 MFMA with fp32 accumulation; P and dS
// enter the second products as bf16.  Q, K, V, dO tiles move global -> LDS
// by buffer_load ... lds (rows past the sequence end read as zero), double
// buffered, two workgroups per CU; no floating-point atomics anywhere.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kThreads = 256;
constexpr int kRowBytes = kHeadDim * 2;        // 256 B per bf16 row
constexpr int kTileBytes = kTile * kRowBytes;  // 16 KB per 64-row tile
constexpr float kLog2e = 1.4426950408889634f;

typedef __attribute__((__vector_size__(4 * sizeof(short)))) short i16x4;
typedef const __attribute__((address_space(4))) int32_t* list_ptr;
typedef const __attribute__((address_space(4))) uint32_t* bits_ptr;

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// Two floats to packed bf16, round to nearest even (one v_cvt_pk_bf16_f32).
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
__device__ __forceinline__ uint32_t cvt_bf16x2(float lo, float hi) {
  const bf16x2_t t = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, t);
}

// Work item of workgroup `slot` among G: each XCD (slot % 8) walks runs of
// 64 consecutive items, so tiles whose operands overlap share that XCD's L2;
// the slots of the last partial group keep their own item.
__device__ __forceinline__ int xcd_item(int slot, int G) {
  constexpr int kRunB = 64, kGroup = 8 * kRunB;
  if (slot >= (G / kGroup) * kGroup) return slot;
  const int r = slot >> 3;
  return (r / kRunB) * kGroup + (slot & 7) * kRunB + r % kRunB;
}

// 16-byte chunk c of tile row r sits at slot c ^ h(r), h(r) = 4 (r % 4) +
// (r / 4) % 4: a permutation of r % 16, so the row reads (16 rows, one chunk
// per pass of a 16-byte read) fall in 16 different bank groups, and the two
// bits 4 (r % 4) differ across 4 consecutive rows, so the transposed reads
// (4 rows x 4 consecutive chunks per half-wave) do too.  The plain r % 16
// served the row reads only: the transposed reads met 4-way bank conflicts.
__device__ __forceinline__ int swz(int row, int c) {
  return c ^ (((row & 3) << 2) | ((row >> 2) & 3));
}

// Row fragment (A or B operand of a 32x32x16 product over the 128 channels):
// tile row `row`, channels 16 ks + 8 g .. +7.
__device__ __forceinline__ bf16x8 row_frag(const uint8_t* t, int row, int ks, int g) {
  return as_bf16x8(*reinterpret_cast<const u32x4*>(t + row * kRowBytes + swz(row, 2 * ks + g) * 16));
}

// A lane's 16 values packed as the bf16 B operand of the two 16-deep
// k-steps that follow (registers 8 cs .. 8 cs + 7 -> step cs).
__device__ __forceinline__ void pack_b(const float (&x)[16], bf16x8 (&pk)[2]) {
#pragma unroll
  for (int cs = 0; cs < 2; ++cs) {
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = cvt_bf16x2(x[8 * cs + 2 * e], x[8 * cs + 2 * e + 1]);
    pk[cs] = __builtin_bit_cast(bf16x8, w);
  }
}

struct BwdParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* o;
  const uint16_t* dout;
  const float* lse;
  const int32_t* idx;
  const int32_t* cnt;
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  float* dvec;      // D [B*H][N]
  uint32_t* bits;   // [B*H][nb][nw]
  Strides qs, ks, vs, os;
  int kmax, H, N, block, nb, nw, ntiles;
  float tau;
  Shape cs;  // causal window (chunk 0: none) and N
};

// ---- D = rowsum(dO o O) -------------------------------------------------
__global__ __launch_bounds__(kThreads) void bwd_dot_kernel(BwdParams p) {
  const int64_t tok = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);  // token of this head
  const int c = threadIdx.x & 15;
  const int bh = blockIdx.y;
  if (tok >= p.N) return;
  const int b = bh / p.H, h = bh - b * p.H;
  const int64_t base = b * p.os.b + h * p.os.h + tok * p.os.n + 8 * c;
  const u32x4 x = ld16(p.o + base), y = ld16(p.dout + base);
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    s = fmaf(bf16_lo(x[e]), bf16_lo(y[e]), s);
    s = fmaf(bf16_hi(x[e]), bf16_hi(y[e]), s);
  }
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) s += __shfl_xor(s, o, 16);
  if (c == 0) p.dvec[(int64_t)bh * p.N + tok] = s;
}

// ---- transposed selection bitmap ----------------------------------------
__global__ __launch_bounds__(kThreads) void bwd_bits_clear_kernel(uint32_t* bits, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i < n) bits[i] = 0u;
}

__global__ __launch_bounds__(kThreads) void bwd_bits_set_kernel(BwdParams p) {
  const int i = blockIdx.x * 4 + (threadIdx.x >> 6);  // query block of head blockIdx.y
  const int bh = blockIdx.y;
  if (i >= p.nb) return;
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)bh * p.nb + i;
  const int c = min(max(p.cnt[r], 0), p.kmax);
  for (int t = lane; t < c; t += kWave) {
    const int j = p.idx[r * p.kmax + t];
    if (j >= 0 && j < p.nb)
      atomicOr(&p.bits[((int64_t)bh * p.nb + j) * p.nw + (i >> 5)], 1u << (i & 31));
  }
}

// ---- copy pipeline ---------------------------------------------------------
// Tiles of 64 rows x 256 bytes move global -> LDS with buffer_load ... lds
// (issued from inline asm, so every wait on them is explicit): each wave
// moves rows 16 w .. 16 w + 15 in 4 instructions of 4 rows, lane l landing
// in slot l % 16 of its row, i.e. fetching the logical chunk that swz() puts
// there.  Rows past the resource range (the sequence end) read zero.
struct TileDma {
  uint32_t off[4];  // per-lane byte offsets within a tile (row stride applied)
};
__device__ __forceinline__ TileDma tile_dma(uint32_t row_bytes) {
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  TileDma t;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int row = 16 * w + 4 * i + (l >> 4);
    t.off[i] = (uint32_t)row * row_bytes + (uint32_t)swz(row, l & 15) * 16u;
  }
  return t;
}
__device__ __forceinline__ void dma_tile(uint8_t* dst, __amdgpu_buffer_rsrc_t r, const TileDma& t,
                                         uint32_t soff) {
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t base = lds_addr(dst) + (uint32_t)(16 * w) * kRowBytes;
#pragma unroll
  for (int i = 0; i < 4; ++i) dma16(base + 4 * i * kRowBytes, r, t.off[i], soff);
}
__device__ __forceinline__ void wait_vm0() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x0F70);
}
__device__ __forceinline__ void wait_vm8() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0x0F78);
}
__device__ __forceinline__ void wait_lgkm0() {
  __builtin_amdgcn_sched_barrier(0);
  __builtin_amdgcn_s_waitcnt(0xC07F);
}

// Start row of the n-th 64-key tile of a query block's list (skipping
// entries out of range and sub-tiles past the end), or N when exhausted.
__device__ __forceinline__ int list_tile(list_ptr list, int n, int total, int spb, int block,
                                         int nb, int N, int* next) {
  for (; n < total; ++n) {
    const int e = n >> (spb - 1);  // spb (sub-tiles per block) is 1 or 2
    const int j = list[e];
    if (j < 0 || j >= nb) continue;
    const int st = j * block + (n - (e << (spb - 1))) * kTile;
    if (st < N) {
      *next = n + 1;
      return st;
    }
  }
  *next = total;
  return N;
}

constexpr int kPBlock = 2048;  // one P or dS block of the dK/dV kernel

// Lane id read afresh, so that offsets derived from it are recomputed where
// they are used instead of being held in registers across the loop.
__device__ __forceinline__ int fresh_lane() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// Transposed reads (ds_read_b64_tr_b16) of the 16 rows r16.. (r16 a multiple
// of 16) of a 64-row tile: lane 16 G + 4 e + q reads the 8 bytes of row
// r16 + 8 hf + 4 (G >> 1) + e at channels 32 dtg + 16 (G & 1) + 4 q, so that
// lane l holds channel 32 dtg + (l & 31) of rows r16 + 4 g + {0..3} (hf = 0)
// and r16 + 8 + 4 g + {0..3} (hf = 1): an A operand over those 16 rows.
// The row's swizzle depends on row & 15 only, so the lane's byte offset is
// the same for every r16.
__device__ __forceinline__ uint32_t trans_off(int lane, int hf, int dtg) {
  const int G = lane >> 4, e4 = (lane >> 2) & 3, q4 = lane & 3;
  const int row = 8 * hf + 4 * (G >> 1) + e4;
  const int lc = 4 * dtg + 2 * (G & 1) + (q4 >> 1);
  return (uint32_t)(row * kRowBytes + swz(row, lc) * 16 + (q4 & 1) * 8);
}
__device__ __forceinline__ u32x2 tr_read(const uint8_t* p) {
  const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p);
  return __builtin_bit_cast(u32x2, v);
}
__device__ __forceinline__ bf16x8 tr_pair(const uint8_t* p0, const uint8_t* p1) {
  const u32x2 a = tr_read(p0), b = tr_read(p1);
  const u32x4 f = {a[0], a[1], b[0], b[1]};
  return as_bf16x8(f);
}

// P and dS: byte offset of the 8-byte unit u (keys 4u..4u+3 of key half kh)
// of query row `row` (0..63).
__device__ __forceinline__ int p_off(int kh, int row, int u) {
  const int qq = row & 31;
  return (kh + 2 * (row >> 5)) * kPBlock + qq * 64 + 8 * (u ^ ((qq >> 2) & 7));
}
// The same transposed read from a P / dS buffer: lane l gets key
// 32 kh + (l & 31) of the rows r16 + 8 hf + 4 g + {0..3} (a B operand in the
// k order of trans_off).  Offset for r16 with bit 4 = b4, before adding
// (r16 >> 5) * 2 kPBlock + b4 * 16 * 64.
__device__ __forceinline__ uint32_t ptr_off(int lane, int hf, int b4, int kh) {
  const int G = lane >> 4, e4 = (lane >> 2) & 3, q4 = lane & 3;
  const int qq = 16 * b4 + 8 * hf + 4 * (G >> 1) + e4;
  return (uint32_t)(p_off(kh, qq, 4 * (G & 1) + q4) - b4 * 16 * 64);
}

// ---- dQ -------------------------------------------------------------------
// Two workgroups per CU (64 KB of LDS each): the Q and dO fragments of the
// wave's query rows are held in registers, K and V tiles are double-buffered,
// and the copies of tile n + 2 are issued once every wave is done with tile n.
__global__ __launch_bounds__(kThreads, 2) void bwd_dq_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t kb0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t kb1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vb0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vb1[kTileBytes];

  const int item = xcd_item((int)blockIdx.x, (int)gridDim.x);
  const int bh = item / p.ntiles;
  const int qt = item - bh * p.ntiles;
  const int b = bh / p.H, h = bh - b * p.H;
  const int q0 = qt * kTile;
  const int iblk = q0 / p.block;
  const int spb = p.block / kTile;
  const list_ptr list = (list_ptr)(p.idx + ((int64_t)bh * p.nb + iblk) * p.kmax);
  const int c = min(max(p.cnt[(int64_t)bh * p.nb + iblk], 0), p.kmax);
  const int total = c * spb;

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rh = wave & 1, kh = wave >> 1;
  const int g = lane >> 5, l32 = lane & 31;

  const uint32_t qst = (uint32_t)p.qs.n * 2, kst = (uint32_t)p.ks.n * 2, vst = (uint32_t)p.vs.n * 2,
                 ost = (uint32_t)p.os.n * 2;
  const auto kr = make_rsrc(p.k + b * p.ks.b + h * p.ks.h, (uint32_t)(p.N - 1) * kst + 256u);
  const auto vr = make_rsrc(p.v + b * p.vs.b + h * p.vs.h, (uint32_t)(p.N - 1) * vst + 256u);
  const TileDma kd = tile_dma(kst), vd = tile_dma(vst);

  // this lane's query row: its LSE (log2 units) and D, loaded and waited for
  // before any copy is issued (a later wait for them would drain the copies)
  const int qtok = q0 + rh * 32 + l32;
  // allowed keys [key_lo, key_hi) of the lane's query (causal window and
  // sequence end); a key tile needs the per-score mask unless it lies in
  // every row's range: [lo of the tile's last row, hi of its first)
  const int key_lo = causal_lo(p.cs, min(qtok, p.N - 1));
  const int key_hi = causal_hi(p.cs, min(qtok, p.N - 1));
  const int tile_lo = causal_lo(p.cs, min(q0 + kTile - 1, p.N - 1));
  const int tile_hi = causal_hi(p.cs, q0);
  float lse2, dq_d;
  {
    const int qc = min(qtok, p.N - 1);
    lse2 = p.lse[(int64_t)bh * p.N + qc];
    dq_d = p.dvec[(int64_t)bh * p.N + qc];
    asm volatile("" : "+v"(lse2), "+v"(dq_d));
    lse2 *= kLog2e;
  }
  const float c2 = p.tau * kLog2e;

  // prologue: Q through kb1, dO through vb1, tiles 0 and 1 of the list
  int nx = 0;
  int s0 = list_tile(list, nx, total, spb, p.block, p.nb, p.N, &nx);
  int s1 = list_tile(list, nx, total, spb, p.block, p.nb, p.N, &nx);
  {
    const auto qr = make_rsrc(p.q + b * p.qs.b + h * p.qs.h, (uint32_t)(p.N - 1) * qst + 256u);
    const auto dr = make_rsrc(p.dout + b * p.os.b + h * p.os.h, (uint32_t)(p.N - 1) * ost + 256u);
    dma_tile(kb1, qr, tile_dma(qst), (uint32_t)q0 * qst);
    dma_tile(vb1, dr, tile_dma(ost), (uint32_t)q0 * ost);
  }
  dma_tile(kb0, kr, kd, (uint32_t)s0 * kst);
  dma_tile(vb0, vr, vd, (uint32_t)s0 * vst);
  wait_vm8();  // Q and dO landed (this wave's rows)
  barrier_keep_loads();
  bf16x8 qf[8], df[8];  // B operands: this lane's query row of Q and dO
  {
    const int qrow = rh * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      qf[ks] = row_frag(kb1, qrow, ks, g);
      df[ks] = row_frag(vb1, qrow, ks, g);
    }
  }
  wait_lgkm0();
  barrier_keep_loads();  // kb1, vb1 free
  dma_tile(kb1, kr, kd, (uint32_t)s1 * kst);
  dma_tile(vb1, vr, vd, (uint32_t)s1 * vst);
  wait_vm8();  // tile 0 landed (this wave's rows); tile 1 may still fly
  barrier_keep_loads();

  f32x16 acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[dt][r] = 0.f;

  // One tile from buffers (kt, vt), which every wave sees landed; once every
  // wave is done reading them and the next tile has landed (one barrier) they
  // receive the tile two ahead, whose start is returned.
  auto step = [&](uint8_t* kt, uint8_t* vt, int st) {
    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.f;
    const int ln = fresh_lane(), g1 = ln >> 5;
    const int krow = kh * 32 + (ln & 31);
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(kt, krow, ks, g1), qf[ks], s, 0, 0, 0);
    __builtin_amdgcn_sched_barrier(0);  // bound the fragments in flight
#pragma unroll
    for (int ks = 0; ks < 8; ++ks)
      dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(vt, krow, ks, g1), df[ks], dp, 0, 0, 0);
    // lane: query qtok, keys st + kh*32 + 8(r>>2) + 4g + (r&3); P = 0 for
    // keys outside the query's range, set after the exponential (a row
    // without any allowed key has LSE = -inf and meets only tiles that take
    // the mask, where all its keys are masked)
    float pr[16], ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) pr[r] = __builtin_amdgcn_exp2f(fmaf(s[r], c2, -lse2));
    if (st + kTile > tile_hi || st < tile_lo) {  // wave-uniform
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = st + kh * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
        if (key < key_lo || key >= key_hi) pr[r] = 0.f;
      }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) ds[r] = pr[r] * (dp[r] - dq_d);
    bf16x8 pk[2];
    pack_b(ds, pk);
    __builtin_amdgcn_sched_barrier(0);
    // dQ^T += K^T dS^T, the K^T fragments (channels 32 dt.., keys 32 kh +
    // 16 cs..) read and used in two halves to bound the registers they hold
    {
      const int ln2 = fresh_lane();
#pragma unroll
      for (int hd = 0; hd < 2; ++hd) {
        bf16x8 kf[2][2];
#pragma unroll
        for (int d2 = 0; d2 < 2; ++d2) {
          const int dt = 2 * hd + d2;
          const uint32_t o0 = trans_off(ln2, 0, dt), o1 = trans_off(ln2, 1, dt);
#pragma unroll
          for (int cs = 0; cs < 2; ++cs) {
            const uint8_t* base = kt + (kh * 32 + 16 * cs) * kRowBytes;
            kf[d2][cs] = tr_pair(base + o0, base + o1);
          }
        }
#pragma unroll
        for (int d2 = 0; d2 < 2; ++d2)
#pragma unroll
          for (int cs = 0; cs < 2; ++cs)
            acc[2 * hd + d2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[d2][cs], pk[cs],
                                                                       acc[2 * hd + d2], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    wait_lgkm0();
    wait_vm0();            // this wave's rows of the next tile landed
    barrier_keep_loads();  // every wave is done reading kt / vt; the next tile is whole
    const int s2 = list_tile(list, nx, total, spb, p.block, p.nb, p.N, &nx);
    dma_tile(kt, kr, kd, (uint32_t)s2 * kst);
    dma_tile(vt, vr, vd, (uint32_t)s2 * vst);
    return s2;
  };
  // tile n sits in buffer n % 2; (st, stn) = starts of tiles n, n + 1
  int st = s0, stn = s1;
  while (st < p.N) {
    const int s2 = step(kb0, vb0, st);
    st = stn;
    stn = s2;
    if (st >= p.N) break;
    const int s3 = step(kb1, vb1, st);
    st = stn;
    stn = s3;
  }
  wait_vm0();
  barrier_keep_loads();

  // sum the two key halves, scale by tau, store
  float* mrg = reinterpret_cast<float*>(rh ? vb0 : kb0);  // 64 x 64 floats per row-half
  if (kh == 1) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mrg[(dt * 16 + r) * kWave + lane] = acc[dt][r];
  }
  __syncthreads();
  if (kh == 0 && qtok < p.N) {
    uint16_t* out = p.dq + b * p.qs.b + h * p.qs.h + (int64_t)qtok * p.qs.n;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        float x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          x[r] = p.tau * (acc[dt][4 * jq + r] + mrg[(dt * 16 + 4 * jq + r) * kWave + lane]);
        u32x2 w;
        w[0] = cvt_bf16x2(x[0], x[1]);
        w[1] = cvt_bf16x2(x[2], x[3]);
        *reinterpret_cast<u32x2*>(out + dt * 32 + 8 * jq + 4 * g) = w;
      }
  }
}

// ---- dK, dV ---------------------------------------------------------------
// One workgroup per 64-key tile (two per CU: 80 KB of LDS, at most 256
// registers a lane); the query tiles of the query blocks that selected its
// key block (set bits of its bitmap row, ascending) stream through
// double-buffered Q and dO tiles, the copies of tile n + 2 issued once every
// wave is done with tile n.  Each step has two phases:
//  1. wave (kh, qh): S^T = K Q^T and dP^T = V dO^T for keys 32 kh.. and
//     query rows 32 qh.. (K, V fragments held in registers), so a lane holds
//     one query row and needs only its LSE and D; P and dS go to LDS as bf16;
//  2. wave (kh, ch): dV^T += dO^T P and dK^T += Q^T dS for keys 32 kh.. and
//     channels 64 ch.., over all 64 rows of the tile (dO^T, Q^T, P and dS by
//     transposed LDS reads).
// P and dS are kept in four 2 KB blocks, one per phase-1 wave (kh, qh): 32
// query rows of 64 B (32 keys), 8-byte unit u of row r at slot
// u ^ ((r >> 2) & 7), conflict-free both for the row writes of phase 1 and
// the transposed reads of phase 2.
__global__ __launch_bounds__(kThreads, 2) void bwd_dkdv_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t qb0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t qb1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t ob0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t ob1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t pbuf[4 * kPBlock];
  __shared__ __attribute__((aligned(1024))) uint8_t sbuf[4 * kPBlock];

  const int item = xcd_item((int)blockIdx.x, (int)gridDim.x);
  const int bh = item / p.ntiles;
  const int kt0 = item - bh * p.ntiles;
  const int b = bh / p.H, h = bh - b * p.H;
  const int k0 = kt0 * kTile;
  const int jblk = k0 / p.block;
  const int spb = p.block / kTile;
  const bits_ptr row_bits = (bits_ptr)(p.bits + ((int64_t)bh * p.nb + jblk) * p.nw);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kh = wave & 1, hh = wave >> 1;  // phase 1: query half hh, phase 2: channel half hh
  const int g = lane >> 5, l32 = lane & 31;

  const uint32_t qst = (uint32_t)p.qs.n * 2, ost = (uint32_t)p.os.n * 2;
  const auto qr = make_rsrc(p.q + b * p.qs.b + h * p.qs.h, (uint32_t)(p.N - 1) * qst + 256u);
  const auto dr = make_rsrc(p.dout + b * p.os.b + h * p.os.h, (uint32_t)(p.N - 1) * ost + 256u);
  const TileDma qd = tile_dma(qst), od = tile_dma(ost);
  const float* lse_h = p.lse + (int64_t)bh * p.N;
  const float* d_h = p.dvec + (int64_t)bh * p.N;

  // Cursor over the query tiles: set bits of the bitmap row (query blocks,
  // ascending), then the block's 64-row sub-tiles; N once exhausted.
  int cw = 0, ci = -1, csub = 0;
  uint32_t cword = p.nw > 0 ? row_bits[0] : 0u;
  auto next_start = [&]() {
    if (ci >= 0 && ++csub < spb) {
      const int st = ci * p.block + csub * kTile;
      if (st < p.N) return st;
    }
    while (cword == 0u && cw + 1 < p.nw) cword = row_bits[++cw];
    if (cword == 0u) return p.N;
    ci = 32 * cw + __builtin_ctz(cword);
    cword &= cword - 1u;
    csub = 0;
    return ci * p.block;  // i < nb, so this start is < N
  };
  // LSE and D of this lane's phase-1 query row of the tile starting at st
  // (the row clamped into the sequence; see to_log2 for rows past its end)
  auto load_vec = [&](int st, float& lv, float& dv) {
    const int tc = min(st + hh * 32 + l32, p.N - 1);
    lv = lse_h[tc];
    dv = d_h[tc];
  };
  // LSE in log2 units, +inf for rows past the end (P = 0 there)
  auto to_log2 = [&](int st, float lv) {
    return st + hh * 32 + l32 < p.N ? lv * kLog2e : INFINITY;
  };

  // K and V fragments of this lane's key (A operands of S^T and dP^T)
  const int key = k0 + kh * 32 + l32;
  bf16x8 kf[8], vf[8];
  {
    const uint16_t* kp = p.k + b * p.ks.b + h * p.ks.h + (int64_t)min(key, p.N - 1) * p.ks.n;
    const uint16_t* vp = p.v + b * p.vs.b + h * p.vs.h + (int64_t)min(key, p.N - 1) * p.vs.n;
    const u32x4 z = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      kf[ks] = as_bf16x8(key < p.N ? ld16(kp + 16 * ks + 8 * g) : z);
      vf[ks] = as_bf16x8(key < p.N ? ld16(vp + 16 * ks + 8 * g) : z);
    }
  }
  const int s0 = next_start();
  const int s1 = next_start();
  float lse2, dd;
  load_vec(s0, lse2, dd);
  asm volatile("" : "+v"(lse2), "+v"(dd) : "v"(kf[0]), "v"(kf[7]), "v"(vf[0]), "v"(vf[7]));
  lse2 = to_log2(s0, lse2);
  dma_tile(qb0, qr, qd, (uint32_t)s0 * qst);
  dma_tile(ob0, dr, od, (uint32_t)s0 * ost);
  dma_tile(qb1, qr, qd, (uint32_t)s1 * qst);
  dma_tile(ob1, dr, od, (uint32_t)s1 * ost);
  wait_vm8();  // tile 0 landed (this wave's rows); tile 1 may still fly
  barrier_keep_loads();

  const float c2 = p.tau * kLog2e;
  // phase 2: wave (mat, hh) accumulates dV^T (mat 0) or dK^T / tau (mat 1)
  // for channels 64 hh + 32 dt .. and keys 32 kb ..
  const int mat = wave & 1;
  f32x16 acc[2][2];
#pragma unroll
  for (int dt = 0; dt < 2; ++dt)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[dt][kb][r] = 0.f;

  // One query tile from (qt, ot) starting at st, which every wave sees
  // landed; stn starts the next one.  Once every wave is done reading
  // (qt, ot) and the next tile has landed (one barrier) they receive the tile
  // two ahead, whose start is returned.
  auto step = [&](uint8_t* qt, uint8_t* ot, int st, int stn) {
    float lsen, ddn;
    load_vec(stn, lsen, ddn);  // waited for before the next copies are issued
    // phase 1: lane holds query row 32 hh + l32, keys 32 kh + 8(r>>2) + 4g + (r&3)
    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.f;
    {
      const int ln = fresh_lane(), g1 = ln >> 5;
      const int qrow = hh * 32 + (ln & 31);
      // the query's allowed keys; the key tile needs the per-score mask
      // unless it lies in every row's range of this query tile
      const int qc = min(st + qrow, p.N - 1);
      const int key_lo = causal_lo(p.cs, qc), key_hi = causal_hi(p.cs, qc);
      const bool edge = k0 + kTile > causal_hi(p.cs, st) ||
                        k0 < causal_lo(p.cs, min(st + kTile - 1, p.N - 1));
#pragma unroll
      for (int ks = 0; ks < 8; ++ks)
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks], row_frag(qt, qrow, ks, g1), s, 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int ks = 0; ks < 8; ++ks)
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[ks], row_frag(ot, qrow, ks, g1), dp, 0, 0,
                                                     0);
      float pa[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) pa[r] = __builtin_amdgcn_exp2f(fmaf(s[r], c2, -lse2));
      if (edge) {  // wave-uniform
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + kh * 32 + 8 * (r >> 2) + 4 * g1 + (r & 3);
          if (key < key_lo || key >= key_hi) pa[r] = 0.f;
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float pv[4], dv[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          pv[e] = pa[4 * i + e];
          dv[e] = pv[e] * (dp[4 * i + e] - dd);
        }
        const int off = p_off(kh, qrow, 2 * i + g1);
        u32x2 wp, wd;
        wp[0] = cvt_bf16x2(pv[0], pv[1]);
        wp[1] = cvt_bf16x2(pv[2], pv[3]);
        wd[0] = cvt_bf16x2(dv[0], dv[1]);
        wd[1] = cvt_bf16x2(dv[2], dv[3]);
        *reinterpret_cast<u32x2*>(pbuf + off) = wp;
        *reinterpret_cast<u32x2*>(sbuf + off) = wd;
      }
    }
    wait_lgkm0();
    barrier_keep_loads();  // P and dS of the whole tile in LDS
    // phase 2: wave (mat, hh): dV^T += dO^T P (mat 0) or dK^T += Q^T dS (mat
    // 1) for channels 64 hh .. and all 64 keys (MFMA output [dt][kb]: lane
    // holds key 32 kb + l32, channels 64 hh + 32 dt + 8(r>>2) + 4g + (r&3));
    // each step reads 2 A and 2 B fragments for 4 MFMAs
    {
      const int ln = fresh_lane();
      uint32_t to[2][2], po[2][2];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          to[hf][x] = trans_off(ln, hf, 2 * hh + x);
          po[hf][x] = ptr_off(ln, hf, x, 0);
        }
      const uint8_t* at = mat ? qt : ot;        // A: Q^T or dO^T
      const uint8_t* bt = mat ? sbuf : pbuf;    // B: dS or P
#define PFRAG(buf, r16)                                                                     \
  tr_pair(buf + ((r16) >> 5) * 2 * kPBlock + ((r16)&16) * 64 + po[0][((r16) >> 4) & 1],     \
          buf + ((r16) >> 5) * 2 * kPBlock + ((r16)&16) * 64 + po[1][((r16) >> 4) & 1])
#define TFRAG(t, r16, dt) tr_pair(t + (r16)*kRowBytes + to[0][dt], t + (r16)*kRowBytes + to[1][dt])
#pragma unroll
      for (int r16 = 0; r16 < kTile; r16 += 16) {
        bf16x8 af[2], bf[2];
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          af[x] = TFRAG(at, r16, x);
          bf[x] = PFRAG(bt + x * kPBlock, r16);  // key half x: block (x, row half)
        }
#pragma unroll
        for (int dt = 0; dt < 2; ++dt)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
            acc[dt][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[dt], bf[kb], acc[dt][kb], 0,
                                                                  0, 0);
      }
#undef PFRAG
#undef TFRAG
    }
    wait_lgkm0();
    // the loads of the next tile's LSE and D complete here, before the copies
    // (a wait for them after the copies would wait for the copies too), and
    // so does this wave's share of the next tile
    asm volatile("" : "+v"(lsen), "+v"(ddn));
    wait_vm0();
    barrier_keep_loads();  // every wave is done reading qt / ot / pbuf / sbuf; next tile whole
    const int s2 = next_start();
    dma_tile(qt, qr, qd, (uint32_t)s2 * qst);
    dma_tile(ot, dr, od, (uint32_t)s2 * ost);
    lse2 = to_log2(stn, lsen);
    dd = ddn;
    return s2;
  };
  int st = s0, stn = s1;
  while (st < p.N) {
    const int s2 = step(qb0, ob0, st, stn);
    st = stn;
    stn = s2;
    if (st >= p.N) break;
    const int s3 = step(qb1, ob1, st, stn);
    st = stn;
    stn = s3;
  }
  wait_vm0();

  // store dV = acc (mat 0) or dK = tau * acc (mat 1): lane holds key
  // 32 kb + l32, 4 channels at a time
  const float sc = mat ? p.tau : 1.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int key2 = k0 + 32 * kb + l32;
    if (key2 >= p.N) continue;
    uint16_t* out = mat ? p.dk + b * p.ks.b + h * p.ks.h + (int64_t)key2 * p.ks.n + 64 * hh
                        : p.dv + b * p.vs.b + h * p.vs.h + (int64_t)key2 * p.vs.n + 64 * hh;
#pragma unroll
    for (int dt = 0; dt < 2; ++dt)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        u32x2 w;
        w[0] = cvt_bf16x2(sc * acc[dt][kb][4 * jq], sc * acc[dt][kb][4 * jq + 1]);
        w[1] = cvt_bf16x2(sc * acc[dt][kb][4 * jq + 2], sc * acc[dt][kb][4 * jq + 3]);
        *reinterpret_cast<u32x2*>(out + dt * 32 + 8 * jq + 4 * g) = w;
      }
  }
}

}  // namespace

size_t bwd_workspace_bytes(const Shape& s) {
  const size_t nw = (size_t)(s.nb + 31) / 32;
  return (size_t)s.B * s.H * s.N * sizeof(float) +
         (size_t)s.B * s.H * s.nb * nw * sizeof(uint32_t) + 256;
}

hipError_t launch_bwd(const Shape& s, const BwdIn& in, void* ws, hipStream_t stream) {
  BwdParams p{};
  p.q = static_cast<const uint16_t*>(in.q);
  p.k = static_cast<const uint16_t*>(in.k);
  p.v = static_cast<const uint16_t*>(in.v);
  p.o = static_cast<const uint16_t*>(in.o);
  p.dout = static_cast<const uint16_t*>(in.dout);
  p.lse = in.lse;
  p.idx = in.idx;
  p.cnt = in.cnt;
  p.dq = static_cast<uint16_t*>(in.dq);
  p.dk = static_cast<uint16_t*>(in.dk);
  p.dv = static_cast<uint16_t*>(in.dv);
  p.qs = in.qs;
  p.ks = in.ks;
  p.vs = in.vs;
  p.os = in.os;
  p.kmax = in.kmax;
  p.H = s.H;
  p.N = s.N;
  p.block = s.block;
  p.nb = s.nb;
  p.nw = (s.nb + 31) / 32;
  p.ntiles = (s.N + kTile - 1) / kTile;
  p.tau = in.softmax_scale;
  p.cs = s;
  uint8_t* w = static_cast<uint8_t*>(ws);
  p.dvec = reinterpret_cast<float*>(w);
  const size_t dbytes = ((size_t)s.B * s.H * s.N * sizeof(float) + 255) / 256 * 256;
  p.bits = reinterpret_cast<uint32_t*>(w + dbytes);
  const int bh = s.B * s.H;
  const int64_t nbits = (int64_t)bh * s.nb * p.nw;
  bwd_dot_kernel<<<dim3((unsigned)((s.N + 15) / 16), (unsigned)bh), kThreads, 0, stream>>>(p);
  bwd_bits_clear_kernel<<<(unsigned)((nbits + kThreads - 1) / kThreads), kThreads, 0, stream>>>(
      p.bits, nbits);
  bwd_bits_set_kernel<<<dim3((unsigned)((s.nb + 3) / 4), (unsigned)bh), kThreads, 0, stream>>>(p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  bwd_dq_kernel<<<bh * p.ntiles, kThreads, 0, stream>>>(p);
  bwd_dkdv_kernel<<<bh * p.ntiles, kThreads, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace sa

// Backward pass of the block-sparse attention forward (the sparse branch of
// paper §2 Eq. comp-sparse; its gradients serve the Stage-1 training of §4),
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
//    that selected its key block (set bits of its bitmap row, ascending);
//    wave (kh, qh): keys 32 kh.., query rows 32 qh.. of each query tile:
//      S = Q K^T, dP = dO V^T, P and dS per lane,
//      dV^T += dO^T P, dK^T += Q^T dS (dO^T, Q^T by transposed reads);
//    the two query halves are summed at the end.
// Every product is a bf16 32x32x16 MFMA with fp32 accumulation; P and dS
// enter the second products as bf16.  Tiles are staged into LDS by plain
// loads (rows past the sequence end read as zero) between barriers.
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

// 16-byte chunk c of tile row r sits at slot c ^ (r & 15).
__device__ __forceinline__ int swz(int row, int c) { return c ^ (row & 15); }

// Stage rows [r0, r0 + 64) of a bf16 [rows][128] matrix (row stride `st`
// elements) into a 16 KB LDS tile; rows at or past `n` read as zero.
__device__ __forceinline__ void stage_tile(uint8_t* dst, const uint16_t* src, int64_t st, int r0,
                                           int n) {
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int e = threadIdx.x + kThreads * m, row = e >> 4, c = e & 15;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (r0 + row < n) v = ld16(src + (int64_t)(r0 + row) * st + 8 * c);
    *reinterpret_cast<u32x4*>(dst + row * kRowBytes + swz(row, c) * 16) = v;
  }
}

// Row fragment (A or B operand of a 32x32x16 product over the 128 channels):
// tile row `row`, channels 16 ks + 8 g .. +7.
__device__ __forceinline__ bf16x8 row_frag(const uint8_t* t, int row, int ks, int g) {
  return as_bf16x8(*reinterpret_cast<const u32x4*>(t + row * kRowBytes + swz(row, 2 * ks + g) * 16));
}

// Transposed fragments (A operand, rows = the 128 channels, k = 32 tile rows
// starting at `r_half`): lane 16G + 4e + q reads the 8 bytes of row
// r_half + 16 cs + 8 hf + 4 (G >> 1) + e at channels 32 dt + 16 (G & 1) + 4 q;
// lane l then holds channel 32 dt + (l & 31) of rows r_half + 16 cs + 8 hf +
// 4 g + {0..3}, the order in which the MFMA output leaves its 16 values.
__device__ __forceinline__ void trans_frags(const uint8_t* t, int r_half, int lane,
                                            u32x4 (&f)[8]) {
  const int G = lane >> 4, e4 = (lane >> 2) & 3, q4 = lane & 3;
  const int row0 = r_half + 4 * (G >> 1) + e4;
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) {
    const int lc = 4 * dt + 2 * (G & 1) + (q4 >> 1);
    const int half = (q4 & 1) * 8;
#pragma unroll
    for (int cs = 0; cs < 2; ++cs)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        const int row = row0 + 16 * cs + 8 * hf;
        const i16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (__attribute__((address_space(3))) i16x4*)(t + row * kRowBytes + swz(row, lc) * 16 +
                                                       half));
        const u32x2 w = __builtin_bit_cast(u32x2, v);
        f[2 * dt + cs][2 * hf] = w[0];
        f[2 * dt + cs][2 * hf + 1] = w[1];
      }
  }
}

// A lane's 16 values packed as the bf16 B operand of the two 16-deep
// k-steps that follow (registers 8 cs .. 8 cs + 7 -> step cs).
__device__ __forceinline__ void pack_b(const float (&x)[16], bf16x8 (&pk)[2]) {
#pragma unroll
  for (int cs = 0; cs < 2; ++cs) {
    u32x4 w;
#pragma unroll
    for (int e = 0; e < 4; ++e) w[e] = pack_bf16x2(x[8 * cs + 2 * e], x[8 * cs + 2 * e + 1]);
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

// ---- dQ -------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void bwd_dq_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t kt[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t vt[kTileBytes];

  const int bh = blockIdx.x / p.ntiles;
  const int qt = blockIdx.x - bh * p.ntiles;
  const int b = bh / p.H, h = bh - b * p.H;
  const int q0 = qt * kTile;
  const int iblk = q0 / p.block;
  const int spb = p.block / kTile;
  const list_ptr list = (list_ptr)(p.idx + ((int64_t)bh * p.nb + iblk) * p.kmax);
  const int c = min(max(p.cnt[(int64_t)bh * p.nb + iblk], 0), p.kmax);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int rh = wave & 1, kh = wave >> 1;
  const int g = lane >> 5, l32 = lane & 31;
  const uint16_t* qh_ = p.q + b * p.qs.b + h * p.qs.h;
  const uint16_t* kh_ = p.k + b * p.ks.b + h * p.ks.h;
  const uint16_t* vh_ = p.v + b * p.vs.b + h * p.vs.h;
  const uint16_t* doh = p.dout + b * p.os.b + h * p.os.h;

  // Q and dO fragments of this lane's query (B operands), staged through LDS
  bf16x8 qf[8], df[8];
  stage_tile(kt, qh_, p.qs.n, q0, p.N);
  stage_tile(vt, doh, p.os.n, q0, p.N);
  __syncthreads();
  {
    const int row = rh * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      qf[ks] = row_frag(kt, row, ks, g);
      df[ks] = row_frag(vt, row, ks, g);
    }
  }
  const int qtok = q0 + rh * 32 + l32;
  const int qc = min(qtok, p.N - 1);
  const float lse2 = p.lse[(int64_t)bh * p.N + qc] * kLog2e;
  const float dq_d = p.dvec[(int64_t)bh * p.N + qc];
  const float c2 = p.tau * kLog2e;

  f32x16 acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[dt][r] = 0.f;

  for (int n = 0; n < c * spb; ++n) {
    const int j = list[n / spb];
    if (j < 0 || j >= p.nb) continue;                     // uniform
    const int s0 = j * p.block + (n % spb) * kTile;
    if (s0 >= p.N) continue;
    __syncthreads();  // previous tile fully read
    stage_tile(kt, kh_, p.ks.n, s0, p.N);
    stage_tile(vt, vh_, p.vs.n, s0, p.N);
    __syncthreads();
    // S^T (keys x queries) and dP^T
    f32x16 s, dp;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.f;
    const int krow = kh * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(kt, krow, ks, g), qf[ks], s, 0, 0, 0);
      dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(vt, krow, ks, g), df[ks], dp, 0, 0, 0);
    }
    // lane: query qtok, keys s0 + kh*32 + 8(r>>2) + 4g + (r&3)
    float ds[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = s0 + kh * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
      const float pr = key < p.N ? __builtin_amdgcn_exp2f(fmaf(s[r], c2, -lse2)) : 0.f;
      ds[r] = pr * (dp[r] - dq_d);
    }
    bf16x8 pk[2];
    pack_b(ds, pk);
    // dQ^T += K^T dS^T
    u32x4 kf[8];
    trans_frags(kt, kh * 32, lane, kf);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int cs = 0; cs < 2; ++cs)
        acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(kf[2 * dt + cs]), pk[cs],
                                                          acc[dt], 0, 0, 0);
  }

  // sum the two key halves, scale by tau, store
  __syncthreads();
  float* mrg = reinterpret_cast<float*>(rh ? vt : kt);  // 64 x 64 floats per row-half
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
        w[0] = pack_bf16x2(x[0], x[1]);
        w[1] = pack_bf16x2(x[2], x[3]);
        *reinterpret_cast<u32x2*>(out + dt * 32 + 8 * jq + 4 * g) = w;
      }
  }
}

// ---- dK, dV ---------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void bwd_dkdv_kernel(BwdParams p) {
  __shared__ __attribute__((aligned(1024))) uint8_t qt_[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t dt_[kTileBytes];
  __shared__ float lse_s[kTile];
  __shared__ float d_s[kTile];

  const int bh = blockIdx.x / p.ntiles;
  const int kt0 = blockIdx.x - bh * p.ntiles;
  const int b = bh / p.H, h = bh - b * p.H;
  const int k0 = kt0 * kTile;
  const int jblk = k0 / p.block;
  const bits_ptr row_bits = (bits_ptr)(p.bits + ((int64_t)bh * p.nb + jblk) * p.nw);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kh = wave & 1, qh = wave >> 1;
  const int g = lane >> 5, l32 = lane & 31;
  const uint16_t* qh_ = p.q + b * p.qs.b + h * p.qs.h;
  const uint16_t* kh_ = p.k + b * p.ks.b + h * p.ks.h;
  const uint16_t* vh_ = p.v + b * p.vs.b + h * p.vs.h;
  const uint16_t* doh = p.dout + b * p.os.b + h * p.os.h;

  // K and V fragments of this lane's key (B operands of S = Q K^T, dP = dO V^T)
  bf16x8 kf[8], vf[8];
  stage_tile(qt_, kh_, p.ks.n, k0, p.N);
  stage_tile(dt_, vh_, p.vs.n, k0, p.N);
  __syncthreads();
  {
    const int row = kh * 32 + l32;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      kf[ks] = row_frag(qt_, row, ks, g);
      vf[ks] = row_frag(dt_, row, ks, g);
    }
  }
  const float c2 = p.tau * kLog2e;

  f32x16 acck[4], accv[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acck[dt][r] = accv[dt][r] = 0.f;

  const int spb = p.block / kTile;
  for (int w = 0; w < p.nw; ++w) {
    uint32_t word = row_bits[w];
    while (word) {
      const int i = 32 * w + __builtin_ctz(word);  // query block, ascending
      word &= word - 1;
      for (int sub = 0; sub < spb; ++sub) {
        const int r0 = i * p.block + sub * kTile;
        if (r0 >= p.N) break;
        __syncthreads();  // previous query tile fully read
        stage_tile(qt_, qh_, p.qs.n, r0, p.N);
        stage_tile(dt_, doh, p.os.n, r0, p.N);
        if (threadIdx.x < kTile) {
          const int t = r0 + threadIdx.x;
          const bool live = t < p.N;
          lse_s[threadIdx.x] = live ? p.lse[(int64_t)bh * p.N + t] * kLog2e : INFINITY;
          d_s[threadIdx.x] = live ? p.dvec[(int64_t)bh * p.N + t] : 0.f;
        }
        __syncthreads();
        // S (queries x keys) and dP: lane holds key kh*32 + l32, queries
        // qh*32 + 8(r>>2) + 4g + (r&3)
        f32x16 s, dp;
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = dp[r] = 0.f;
        const int qrow = qh * 32 + l32;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) {
          s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(qt_, qrow, ks, g), kf[ks], s, 0, 0,
                                                      0);
          dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(row_frag(dt_, qrow, ks, g), vf[ks], dp, 0,
                                                       0, 0);
        }
        float pv[16], ds[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int ql = qh * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
          const float pr = __builtin_amdgcn_exp2f(fmaf(s[r], c2, -lse_s[ql]));
          pv[r] = pr;
          ds[r] = pr * (dp[r] - d_s[ql]);
        }
        bf16x8 pp[2], pd[2];
        pack_b(pv, pp);
        pack_b(ds, pd);
        u32x4 tf[8];
        trans_frags(dt_, qh * 32, lane, tf);  // dO^T
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int cs = 0; cs < 2; ++cs)
            accv[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(tf[2 * dt + cs]), pp[cs],
                                                               accv[dt], 0, 0, 0);
        trans_frags(qt_, qh * 32, lane, tf);  // Q^T
#pragma unroll
        for (int dt = 0; dt < 4; ++dt)
#pragma unroll
          for (int cs = 0; cs < 2; ++cs)
            acck[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(tf[2 * dt + cs]), pd[cs],
                                                               acck[dt], 0, 0, 0);
      }
    }
  }

  // sum the two query halves, store dK = tau * acck, dV = accv
  __syncthreads();
  float* mk = reinterpret_cast<float*>(kh ? dt_ : qt_);  // 64 x 64 floats per key half
  if (qh == 1) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mk[(dt * 16 + r) * kWave + lane] = acck[dt][r];
  }
  __syncthreads();
  const int key = k0 + kh * 32 + l32;
  if (qh == 0 && key < p.N) {
    uint16_t* out = p.dk + b * p.ks.b + h * p.ks.h + (int64_t)key * p.ks.n;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        float x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          x[r] = p.tau * (acck[dt][4 * jq + r] + mk[(dt * 16 + 4 * jq + r) * kWave + lane]);
        u32x2 w;
        w[0] = pack_bf16x2(x[0], x[1]);
        w[1] = pack_bf16x2(x[2], x[3]);
        *reinterpret_cast<u32x2*>(out + dt * 32 + 8 * jq + 4 * g) = w;
      }
  }
  __syncthreads();
  if (qh == 1) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mk[(dt * 16 + r) * kWave + lane] = accv[dt][r];
  }
  __syncthreads();
  if (qh == 0 && key < p.N) {
    uint16_t* out = p.dv + b * p.vs.b + h * p.vs.h + (int64_t)key * p.vs.n;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        float x[4];
#pragma unroll
        for (int r = 0; r < 4; ++r)
          x[r] = accv[dt][4 * jq + r] + mk[(dt * 16 + 4 * jq + r) * kWave + lane];
        u32x2 w;
        w[0] = pack_bf16x2(x[0], x[1]);
        w[1] = pack_bf16x2(x[2], x[3]);
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

// Fused block-sparse attention forward, bf16 operands, for gfx950.
//
// Computes the sparse branch A_M of compensated sparse attention (paper §2
// Eq. comp-sparse, §4.1): exact softmax attention of each 64-row query tile
// over the union of the key blocks its query block selected.
//
// One workgroup = 4 wavefronts = one 64-row query tile.  Every selected key
// block is walked as 64-key tiles that are staged in LDS (double-buffered,
// K row-major, V transposed so that the PV product reads keys contiguously).
// Wave w owns query rows 32*(w&1)..+31 and keys 32*(w>>1)..+31 of every tile:
//   S^T (32 keys x 32 queries) = K_half . Q_half^T  -- 8 x v_mfma_f32_32x32x16_bf16
//   online softmax in fp32 registers (exp2 with tau*log2(e) folded in)
//   O^T (128 x 32)          += V_half^T . P^T       -- 8 x v_mfma_f32_32x32x16_bf16
// Computing S transposed puts all 16 scores of a lane in one query column,
// so the row statistics are per-lane scalars and the probabilities already
// sit in the B-operand layout of the PV product (no LDS round trip for P).
// The two key-half waves of a row-half keep separate softmax states that are
// merged through LDS at the end.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kThreads = 256;
constexpr int kKRow = kHeadDim + 8;  // LDS K row stride (bf16): 272 B, 16-B aligned
constexpr int kVRow = kTile + 4;     // LDS V^T row stride (bf16): 136 B, 8-B aligned
constexpr int kKBuf = kTile * kKRow;
constexpr int kVBuf = kHeadDim * kVRow;
constexpr int kLdsElems = 2 * kKBuf + 2 * kVBuf;  // 69632 bytes

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
};

// Start row of the n-th 64-key tile of a query block's list, or -1 when the
// list entry is out of range or the sub-tile lies past the sequence end.
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

struct TileRegs {
  u32x4 k[4];
  u32x4 v[4];
};

// Global -> registers for one 64-key tile; rows past N read as zero.
__device__ __forceinline__ void load_tile(TileRegs& r, const uint16_t* kb, const uint16_t* vb,
                                          const Params& p, int start) {
  const int t = threadIdx.x;
  const int chunk = t & 15;
  const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int row = start + (t >> 4) + 16 * m;
    r.k[m] = row < p.N ? ld16(kb + (int64_t)row * p.ks.n + chunk * 8) : zero;
  }
  const int kq = t >> 4;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int row = start + 4 * kq + m;
    r.v[m] = row < p.N ? ld16(vb + (int64_t)row * p.vs.n + chunk * 8) : zero;
  }
}

// Registers -> LDS buffer: K row-major, V transposed (4-key chunks per d row).
__device__ __forceinline__ void store_tile(const TileRegs& r, uint16_t* ks, uint16_t* vt) {
  const int t = threadIdx.x;
  const int chunk = t & 15;
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int row = (t >> 4) + 16 * m;
    st16(ks + row * kKRow + chunk * 8, r.k[m]);
  }
  const int kq = t >> 4;
#pragma unroll
  for (int x = 0; x < 4; ++x) {
    // even channel d = 8*chunk + 2x (low halves), odd channel d + 1 (high halves)
    u32x2 ev, od;
    ev[0] = (r.v[0][x] & 0xffffu) | (r.v[1][x] << 16);
    ev[1] = (r.v[2][x] & 0xffffu) | (r.v[3][x] << 16);
    od[0] = (r.v[0][x] >> 16) | (r.v[1][x] & 0xffff0000u);
    od[1] = (r.v[2][x] >> 16) | (r.v[3][x] & 0xffff0000u);
    const int d = chunk * 8 + 2 * x;
    *reinterpret_cast<u32x2*>(vt + d * kVRow + kq * 4) = ev;
    *reinterpret_cast<u32x2*>(vt + (d + 1) * kVRow + kq * 4) = od;
  }
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__global__ __launch_bounds__(kThreads, 2) void fwd_bf16_kernel(Params p) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[kLdsElems];
  // buffer x: K at lds + x * kKBuf, V^T at lds + 2 * kKBuf + x * kVBuf
  auto ks_buf = [&](int x) { return lds + x * kKBuf; };
  auto vt_buf = [&](int x) { return lds + 2 * kKBuf + x * kVBuf; };

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
  const int rh = wave & 1, kh = wave >> 1;
  const int g = lane >> 5, l32 = lane & 31;

  const uint16_t* kbase = p.k + b * p.ks.b + h * p.ks.h;
  const uint16_t* vbase = p.v + b * p.vs.b + h * p.vs.h;

  // Q fragment (B operand of K.Q^T): query row l32 of this row-half,
  // channels 16*ks + 8*g .. +7.
  bf16x8 qf[8];
  {
    const int row = q0 + rh * 32 + l32;
    const uint16_t* qp = p.q + b * p.qs.b + h * p.qs.h + (int64_t)row * p.qs.n + g * 8;
    const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[s] = as_bf16x8(row < p.N ? ld16(qp + s * 16) : zero);
  }

  f32x16 acc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[dt][r] = 0.f;
  float m2 = -INFINITY;  // running max of tau*log2(e)*logit for this lane's query
  float lsum = 0.f;      // partial sum of exp2 over this lane's keys

  int start = 0;
  int n = next_tile(list, 0, total, spb, p.block, p.nb, p.N, &start);
  TileRegs regs;
  if (n < total) {
    load_tile(regs, kbase, vbase, p, start);
    store_tile(regs, ks_buf(0), vt_buf(0));
  }
  __syncthreads();

  int buf = 0;
  while (n < total) {
    int nstart = 0;
    const int nn = next_tile(list, n + 1, total, spb, p.block, p.nb, p.N, &nstart);
    if (nn < total) load_tile(regs, kbase, vbase, p, nstart);

    // ---- S^T = K_half . Q^T ------------------------------------------------
    f32x16 s;
#pragma unroll
    for (int r = 0; r < 16; ++r) s[r] = 0.f;
    const uint16_t* krow = ks_buf(buf) + (kh * 32 + l32) * kKRow + g * 8;
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
      const bf16x8 kf = as_bf16x8(*reinterpret_cast<const u32x4*>(krow + ks * 16));
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s, 0, 0, 0);
    }
    // lane holds keys kh*32 + 8*(r>>2) + 4*g + (r&3) of query l32
    if (start + kTile > p.N) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = start + kh * 32 + 8 * (r >> 2) + 4 * g + (r & 3);
        if (key >= p.N) s[r] = -INFINITY;
      }
    }

    // ---- online softmax --------------------------------------------------
    float mx = s[0];
#pragma unroll
    for (int r = 1; r < 16; ++r) mx = fmaxf(mx, s[r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
    const float mnew = fmaxf(m2, mx * p.scale_log2);
    const float msafe = mnew == -INFINITY ? 0.f : mnew;
    const float alpha = __builtin_amdgcn_exp2f(m2 - msafe);
    float pv[16];
    float psum = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      pv[r] = __builtin_amdgcn_exp2f(fmaf(s[r], p.scale_log2, -msafe));
      psum += pv[r];
    }
    lsum = lsum * alpha + psum;
    m2 = mnew;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[dt][r] *= alpha;

    // P^T as B operand: k-step c uses registers 8c .. 8c+7 (keys
    // 16c + 4g + {0..3} and 16c + 8 + 4g + {0..3} of the half).
    bf16x8 pk[2];
#pragma unroll
    for (int cs = 0; cs < 2; ++cs)
#pragma unroll
      for (int e = 0; e < 8; ++e) pk[cs][e] = (__bf16)pv[8 * cs + e];

    // ---- O^T += V_half^T . P^T -------------------------------------------
    const uint16_t* vrow = vt_buf(buf) + l32 * kVRow + (kh * 8 + g) * 4;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
#pragma unroll
      for (int cs = 0; cs < 2; ++cs) {
        const uint16_t* vp = vrow + dt * 32 * kVRow + cs * 16;
        const u32x2 lo = *reinterpret_cast<const u32x2*>(vp);
        const u32x2 hi = *reinterpret_cast<const u32x2*>(vp + 8);
        const u32x4 vv = {lo[0], lo[1], hi[0], hi[1]};
        acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(vv), pk[cs], acc[dt], 0, 0, 0);
      }
    }

    if (nn < total) store_tile(regs, ks_buf(buf ^ 1), vt_buf(buf ^ 1));
    __syncthreads();
    buf ^= 1;
    n = nn;
    start = nstart;
  }

  // ---- merge the two key halves, normalise, store ------------------------
  lsum += __shfl_xor(lsum, 32, kWave);
  float* mrg = reinterpret_cast<float*>(lds) + rh * (66 * kWave);
  if (kh == 1) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) mrg[(dt * 16 + r) * kWave + lane] = acc[dt][r];
    mrg[64 * kWave + lane] = m2;
    mrg[65 * kWave + lane] = lsum;
  }
  __syncthreads();
  if (kh == 0) {
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
  const int grid = s.B * s.H * p.ntiles;
  fwd_bf16_kernel<<<grid, kThreads, 0, stream>>>(p);
  return hipGetLastError();
}

}  // namespace sa

// Work scheduling for the fused forward: orders the 64-row query tiles of all
// (batch, head) slices for the hardware dispatcher.
//
// The dispatcher hands workgroups out in blockIdx order as CU slots free up,
// i.e. it is a greedy list scheduler.  Two properties of the order matter:
//  * ragged cost (query blocks keep different numbers of key blocks): tiles
//    are sorted by a cost class, most expensive first (longest-processing-
//    time-first), so short tiles fill the tail of the launch;
//  * locality: within a class, tiles stay in raster order, and blockIdx is
//    remapped so that each XCD (blockIdx % 8 on MI355X) receives runs of
//    consecutive tiles, whose key-block lists overlap and share that XCD's L2.
// The cost classes are floor(log2(key tiles)) so the sort is a 16-bucket
// stable partition computed by one workgroup.
#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kSchedThreads = 1024;
constexpr int kClasses = 16;
constexpr int kXcds = 8;
constexpr int kRun = 64;  // consecutive list positions handed to one XCD

__device__ __forceinline__ int cost_class(int tiles) {
  // 0 for empty tiles; otherwise 1 + floor(log2(tiles)), capped.  Larger = costlier.
  if (tiles <= 0) return 0;
  const int c = 32 - __clz(tiles);
  return c < kClasses ? c : kClasses - 1;
}

// Position in the cost-sorted list that launch slot `b` (of G) takes.
__device__ __forceinline__ int slot_to_pos(int b, int G) {
  const int group = kXcds * kRun;
  const int full = (G / group) * group;
  if (b >= full) return b;
  const int x = b % kXcds, r = b / kXcds;
  return (r / kRun) * group + x * kRun + (r % kRun);
}

// Classes of up to this many tiles are kept in LDS (one byte each) between
// the histogram and the scatter pass; larger launches recompute them.
constexpr int kClassCache = 64 * 1024;

__global__ __launch_bounds__(kSchedThreads) void schedule_kernel(const int32_t* __restrict__ cnt,
                                                                 int kmax, int nb, int ntiles,
                                                                 int block, int G,
                                                                 int32_t* __restrict__ list,
                                                                 int32_t* __restrict__ order) {
  __shared__ int hist[kClasses];
  __shared__ int base[kClasses];
  __shared__ int wave_cnt[kSchedThreads / kWave][kClasses];
  __shared__ uint8_t cls_cache[kClassCache];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  const int spb = block / kTile;
  const bool cached = G <= kClassCache;
  if (t < kClasses) hist[t] = 0;
  __syncthreads();

  auto cls_of = [&](int item) {
    const int bh = item / ntiles, qt = item - bh * ntiles;
    const int c = cnt[(int64_t)bh * nb + (qt * kTile) / block];
    return cost_class(min(max(c, 0), kmax) * spb);
  };

  // Histogram pass: the loads of all items are independent, so they overlap.
  for (int it = t; it < G; it += kSchedThreads) {
    const int c = cls_of(it);
    if (cached) cls_cache[it] = (uint8_t)c;
    atomicAdd(&hist[c], 1);
  }
  __syncthreads();
  if (t == 0) {
    int acc = 0;
    for (int c = kClasses - 1; c >= 0; --c) {  // costliest class first
      base[c] = acc;
      acc += hist[c];
    }
  }
  __syncthreads();

  const uint64_t below = lanes_below_mask();
  for (int c0 = 0; c0 < G; c0 += kSchedThreads) {
    const int it = c0 + t;
    const int cls = it < G ? (cached ? (int)cls_cache[it] : cls_of(it)) : -1;
    int rank = 0;
#pragma unroll
    for (int c = 0; c < kClasses; ++c) {
      const uint64_t m = __ballot(cls == c);
      if (cls == c) rank = __popcll(m & below);
      if (lane == 0) wave_cnt[wave][c] = __popcll(m);
    }
    __syncthreads();
    if (cls >= 0) {
      int pos = base[cls] + rank;
      for (int w = 0; w < wave; ++w) pos += wave_cnt[w][cls];
      list[pos] = it;
    }
    __syncthreads();
    if (t < kClasses) {
      int tot = 0;
      for (int w = 0; w < kSchedThreads / kWave; ++w) tot += wave_cnt[w][t];
      base[t] += tot;
    }
    __syncthreads();
  }
  // list[] is complete; every thread of this single workgroup can read it now.
  __threadfence_block();
  __syncthreads();
  for (int b = t; b < G; b += kSchedThreads) order[b] = list[slot_to_pos(b, G)];
}

}  // namespace

int64_t num_query_tiles(const Shape& s) {
  return (int64_t)s.B * s.H * ((s.N + kTile - 1) / kTile);
}

size_t schedule_workspace_bytes(const Shape& s) {
  return (size_t)num_query_tiles(s) * sizeof(int32_t);
}

hipError_t launch_schedule(const Shape& s, const int32_t* cnt, int kmax, int32_t* order,
                           void* ws, hipStream_t stream) {
  const int ntiles = (s.N + kTile - 1) / kTile;
  const int G = (int)num_query_tiles(s);
  int32_t* list = static_cast<int32_t*>(ws);
  schedule_kernel<<<1, kSchedThreads, 0, stream>>>(cnt, kmax, s.nb, ntiles, s.block, G, list,
                                                   order);
  return hipGetLastError();
}

}  // namespace sa

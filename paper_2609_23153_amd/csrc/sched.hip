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
// The cost classes are floor(log2(key tiles)), so the sort is a 16-bucket
// stable partition (a counting sort), done by three small launches over
// chunks of 1024 tiles: class counts per chunk, one exclusive scan of the
// counts (classes descending, chunks ascending), and a scatter that writes
// every tile straight into its launch slot.
#include <mutex>

#include "common.h"
#include "launch.h"

namespace sa {
namespace {

constexpr int kClasses = 16;
constexpr int kXcds = 8;
constexpr int kRun = 256;          // consecutive list positions handed to one XCD
constexpr int kChunk = 1024;       // tiles per counting / scatter workgroup
constexpr int kSortThreads = 256;  // 4 waves x 4 rounds of 64 tiles
constexpr int kScanThreads = 1024;

__device__ __forceinline__ int cost_class(int tiles) {
  // 0 for empty tiles; otherwise 1 + floor(log2(tiles)), capped.  Larger = costlier.
  if (tiles <= 0) return 0;
  const int c = 32 - __clz(tiles);
  return c < kClasses ? c : kClasses - 1;
}

struct SchedArgs {
  const int32_t* cnt;
  int kmax, nb, ntiles, block, G, chunks;
};

__device__ __forceinline__ int class_of(const SchedArgs& a, int item) {
  const int bh = item / a.ntiles, qt = item - bh * a.ntiles;
  const int c = a.cnt[(int64_t)bh * a.nb + (qt * kTile) / a.block];
  return cost_class(min(max(c, 0), a.kmax) * (a.block / kTile));
}

// Launch slot that takes sorted position `pos` (of G): the inverse of the
// interleave that gives XCD x (slot % 8) runs of kRun consecutive positions;
// the positions of the last partial group keep their own slot.
__device__ __forceinline__ int pos_to_slot(int pos, int G) {
  const int group = kXcds * kRun;
  const int full = (G / group) * group;
  if (pos >= full) return pos;
  const int g = pos / group, rem = pos - g * group;
  const int x = rem / kRun, rr = rem - x * kRun;
  return (g * kRun + rr) * kXcds + x;
}

// counts[chunk][c] = tiles of class c in the chunk.
__global__ __launch_bounds__(kSortThreads) void sched_count_kernel(SchedArgs a,
                                                                   int32_t* __restrict__ counts) {
  __shared__ int wave_cnt[kSortThreads / kWave][kClasses];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  int mine = 0;  // lane c of each wave keeps the wave's count of class c
#pragma unroll
  for (int m = 0; m < kChunk / kSortThreads; ++m) {
    const int it = blockIdx.x * kChunk + m * kSortThreads + t;
    const int cls = it < a.G ? class_of(a, it) : -1;
#pragma unroll
    for (int c = 0; c < kClasses; ++c) {
      const int n = __popcll(__ballot(cls == c));
      if (lane == c) mine += n;
    }
  }
  if (lane < kClasses) wave_cnt[wave][lane] = mine;
  __syncthreads();
  if (t < kClasses) {
    int tot = 0;
#pragma unroll
    for (int w = 0; w < kSortThreads / kWave; ++w) tot += wave_cnt[w][t];
    counts[(int64_t)blockIdx.x * kClasses + t] = tot;
  }
}

// In place: counts[chunk][c] becomes the number of class-c tiles in earlier
// chunks; counts[chunks][c] receives the first sorted position of class c
// (classes in descending order).  One workgroup.
__global__ __launch_bounds__(kScanThreads) void sched_scan_kernel(int chunks,
                                                                  int32_t* __restrict__ counts) {
  __shared__ int wsum[kScanThreads / kWave][kClasses];
  __shared__ int carry[kClasses];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  if (t < kClasses) carry[t] = 0;
  __syncthreads();
  for (int ch0 = 0; ch0 < chunks; ch0 += kScanThreads) {
    const int ch = ch0 + t;
    int v[kClasses], incl[kClasses];
#pragma unroll
    for (int c = 0; c < kClasses; ++c) {
      v[c] = ch < chunks ? counts[(int64_t)ch * kClasses + c] : 0;
      incl[c] = v[c];
    }
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1)
#pragma unroll
      for (int c = 0; c < kClasses; ++c) {
        const int y = __shfl_up(incl[c], o, kWave);
        if (lane >= o) incl[c] += y;
      }
    if (lane == kWave - 1)
#pragma unroll
      for (int c = 0; c < kClasses; ++c) wsum[wave][c] = incl[c];
    __syncthreads();
    if (ch < chunks) {
#pragma unroll
      for (int c = 0; c < kClasses; ++c) {
        int before = carry[c];
        for (int w = 0; w < wave; ++w) before += wsum[w][c];
        counts[(int64_t)ch * kClasses + c] = before + incl[c] - v[c];
      }
    }
    __syncthreads();
    if (t < kClasses) {
      int tot = 0;
      for (int w = 0; w < kScanThreads / kWave; ++w) tot += wsum[w][t];
      carry[t] += tot;
    }
    __syncthreads();
  }
  if (t == 0) {
    int acc = 0;
    for (int c = kClasses - 1; c >= 0; --c) {  // costliest class first
      counts[(int64_t)chunks * kClasses + c] = acc;
      acc += carry[c];
    }
  }
}

// Each tile's sorted position = class start + class-c tiles in earlier chunks
// + class-c tiles before it in this chunk; written to order[slot(position)].
__global__ __launch_bounds__(kSortThreads) void sched_scatter_kernel(
    SchedArgs a, const int32_t* __restrict__ counts, int32_t* __restrict__ order) {
  __shared__ int run[kClasses];
  __shared__ int wave_cnt[kSortThreads / kWave][kClasses];
  const int t = threadIdx.x, lane = t & (kWave - 1), wave = t / kWave;
  if (t < kClasses)
    run[t] = counts[(int64_t)a.chunks * kClasses + t] +
             counts[(int64_t)blockIdx.x * kClasses + t];
  const uint64_t below = lanes_below_mask();
  for (int m = 0; m < kChunk / kSortThreads; ++m) {
    // tiles of round m in index order: wave w holds the w-th 64 of them
    const int it = blockIdx.x * kChunk + m * kSortThreads + t;
    const int cls = it < a.G ? class_of(a, it) : -1;
    int rank = 0;
#pragma unroll
    for (int c = 0; c < kClasses; ++c) {
      const uint64_t msk = __ballot(cls == c);
      if (cls == c) rank = __popcll(msk & below);
      if (lane == c) wave_cnt[wave][c] = __popcll(msk);
    }
    __syncthreads();
    if (cls >= 0) {
      int pos = run[cls] + rank;
      for (int w = 0; w < wave; ++w) pos += wave_cnt[w][cls];
      order[pos_to_slot(pos, a.G)] = it;
    }
    __syncthreads();
    if (t < kClasses) {
      int tot = 0;
#pragma unroll
      for (int w = 0; w < kSortThreads / kWave; ++w) tot += wave_cnt[w][t];
      run[t] += tot;
    }
    __syncthreads();
  }
}

}  // namespace

int64_t num_query_tiles(const Shape& s) {
  return (int64_t)s.B * s.H * ((s.N + kTile - 1) / kTile);
}

size_t schedule_workspace_bytes(const Shape& s) {
  const int64_t chunks = (num_query_tiles(s) + kChunk - 1) / kChunk;
  return (size_t)(chunks + 1) * kClasses * sizeof(int32_t);
}

// ---- allocation-free variant ----------------------------------------------
// The class counters live in one file-scope device array per GPU instead of a
// caller workspace.  In host code `scratch` names a host-side stand-in, not
// device memory: the device address of each GPU's copy is looked up once per
// device (hipGetSymbolAddress with that device current) and only that address
// is handed to the kernels.
namespace {
constexpr int kScratchInts = kStaticScheduleScratchBytes / (int)sizeof(int32_t);
static __device__ __align__(256) int32_t scratch[kScratchInts];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int32_t* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t static_schedule_scratch(int32_t** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = static_cast<int32_t*>(p);
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_schedule(const Shape& s, const int32_t* cnt, int kmax, int32_t* order,
                           void* ws, hipStream_t stream) {
  SchedArgs a;
  a.cnt = cnt;
  a.kmax = kmax;
  a.nb = s.nb;
  a.ntiles = (s.N + kTile - 1) / kTile;
  a.block = s.block;
  a.G = (int)num_query_tiles(s);
  a.chunks = (a.G + kChunk - 1) / kChunk;
  int32_t* counts = static_cast<int32_t*>(ws);
  sched_count_kernel<<<a.chunks, kSortThreads, 0, stream>>>(a, counts);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  sched_scan_kernel<<<1, kScanThreads, 0, stream>>>(a.chunks, counts);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  sched_scatter_kernel<<<a.chunks, kSortThreads, 0, stream>>>(a, counts, order);
  return hipGetLastError();
}

}  // namespace sa

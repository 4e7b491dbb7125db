// Device-side vocabulary shared by the gfx950 kernels of the library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(8 * sizeof(int)))) int i32x8;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2;

constexpr int kHeadDim = 128;   // d handled by every kernel
constexpr int kWave = 64;       // CDNA wavefront width
constexpr int kTile = 64;       // query rows / keys per fwd tile

// Buffer resource over `bytes` bytes from `base`: loads at offsets past the
// end return zero (the hardware range check), without branches.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}
__device__ __forceinline__ u32x4 buf_ld16(__amdgpu_buffer_rsrc_t r, uint32_t off,
                                          uint32_t soff = 0) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, 0));
}

// max of x over the lane pair (l, l ^ 32), through v_permlane32_swap.
__device__ __forceinline__ float pair_max32(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
}

// Global -> LDS copy of 16 bytes per lane (buffer_load_dwordx4 ... lds): lane
// l's bytes land at LDS byte address lds_addr + 16*l; rows past the resource
// range land as zeros.  Issued from inline asm so that the compiler does not
// track it: callers wait (vmcnt) and synchronise explicitly.  The compiler's
// own waits stay correct (they can only become more conservative), and the
// memory clobber keeps program order for every memory access around it.
__device__ __forceinline__ void dma16(uint32_t lds_addr, __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                      uint32_t soff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :: "s"(lds_addr), "v"(voff), "s"(r), "s"(soff)
               : "memory", "m0");
}

// LDS byte address of a __shared__ pointer.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// Workgroup barrier for pipelined LDS staging: unlike __syncthreads() it has
// no release fence, which would wait for every load in flight (vmcnt(0)),
// including global->LDS copies meant to stay in flight across the barrier.
// The caller waits explicitly for the copies the next step reads; the memory
// clobber keeps the compiler from moving memory accesses across.
__device__ __forceinline__ void barrier_keep_loads() { asm volatile("s_barrier" ::: "memory"); }

// 16-byte global load / store (dwordx4) of raw bits.
__device__ __forceinline__ u32x4 ld16(const void* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 round to nearest even (finite inputs).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return f32_to_bf16_rne(lo) | (f32_to_bf16_rne(hi) << 16);
}

// OCP e4m3fn code of y for |y| < 464 (callers scale so that |y| <= 448, up
// to one fp32 rounding): nearest value, ties to even, sign bit kept (so -0
// and tiny negatives give 0x80).  Integer arithmetic on the fp32 fields.
__device__ __forceinline__ uint32_t e4m3_rne(float y) {
  const uint32_t u = __float_as_uint(y);
  const uint32_t sign = (u >> 24) & 0x80u;
  const uint32_t a = u & 0x7fffffffu;
  uint32_t code;
  if (a < 0x3c800000u) {  // |y| < 2^-6: e4m3 subnormal grid of step 2^-9
    code = (uint32_t)__builtin_rintf(__uint_as_float(a) * 512.f);  // 0 .. 8
  } else {
    const uint32_t e = a >> 23;          // fp32 biased exponent (>= 121)
    const uint32_t m3 = (a >> 20) & 7u;  // top 3 mantissa bits
    const uint32_t rem = a & 0xfffffu;
    const uint32_t up = (rem > 0x80000u) || (rem == 0x80000u && (m3 & 1u));
    code = (((e - 120u) << 3) | m3) + up;  // e4m3 exponent bias 7 = fp32 bias 127 - 120
  }
  return sign | code;
}

// Whole-wave reductions through DPP-free cross-lane shuffles.
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, kWave));
  return x;
}
__device__ __forceinline__ int wave_sum(int x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o, kWave);
  return x;
}

__device__ __forceinline__ uint64_t lanes_below_mask() {
  const int lane = threadIdx.x & (kWave - 1);
  return lane == 0 ? 0ull : (~0ull >> (kWave - lane));
}

}  // namespace sa

// Device helpers shared by the libarctopk kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace arc {

constexpr int kWave = 64;

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Load of data the kernel reads exactly once, marked non-temporal so that it
// does not displace reusable lines.  Only for full 16-byte accesses: a
// partial-line non-temporal load loses the rest of the line.
__device__ __forceinline__ float4 stream_load(const float4* p) {
  const f32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

// Store of data nobody reads again in this kernel, marked non-temporal.
__device__ __forceinline__ void stream_store(float4* p, float4 v) {
  const f32x4_t w = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(w, reinterpret_cast<f32x4_t*>(p));
}

// Raw buffer resource (stride 0) over `bytes` bytes from `base`.  Vector
// memory instructions through it are range checked by the hardware on their
// VGPR offset: a load at an offset >= bytes returns zero and a store there is
// dropped.  Offsets are 32-bit byte offsets.
typedef __amdgpu_buffer_rsrc_t buffer_rsrc;
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
constexpr int kBufferDword3 = 0x00020000;  // gfx9-family raw buffer: 32-bit data format
constexpr int kCacheDefault = 0;
constexpr int kCacheNonTemporal = 2;       // nt cache-policy bit on gfx950
// nt with the sc1 bit (device scope): for a stream written once and read by
// later launches only.  For the sketch stage's h stores it measured 0.3-1.4%
// faster than nt alone (1.1B step 9.71 -> 9.56 ms), and without nt slower.
constexpr int kCacheStreamDevice = 2 | 16;

__device__ __forceinline__ buffer_rsrc make_buffer(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           kBufferDword3);
}

template <int kPolicy>
__device__ __forceinline__ float4 buffer_load_f4(buffer_rsrc r, uint32_t off) {
  const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kPolicy);
  return make_float4(__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z),
                     __uint_as_float(v.w));
}

template <int kPolicy>
__device__ __forceinline__ uint2 buffer_load_u2(buffer_rsrc r, uint32_t off) {
  const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, kPolicy);
  return make_uint2(v.x, v.y);
}

template <int kPolicy>
__device__ __forceinline__ void buffer_store_f4(buffer_rsrc r, uint32_t off, float4 v) {
  const u32x4_t w = {__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                     __float_as_uint(v.w)};
  __builtin_amdgcn_raw_buffer_store_b128(w, r, (int)off, 0, kPolicy);
}

// Workgroups are dispatched round-robin over the 8 XCDs of the MI355X (block
// b starts on XCD b % 8).  This bijection of [0, nblocks) hands each XCD one
// contiguous range of blocks (the last nblocks % 8 map to themselves).
__device__ __forceinline__ int64_t xcd_contiguous_block(int64_t b, int64_t nblocks) {
  constexpr int64_t kXcds = 8;
  const int64_t per = nblocks / kXcds;
  return b < per * kXcds ? (b % kXcds) * per + b / kXcds : b;
}

// bf16 halves of a 32-bit word, widened exactly to binary32.
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Order this wave's LDS accesses: everything issued before has completed
// before anything after is issued (LDS rows that only this wave touches).
__device__ __forceinline__ void wave_lds_fence() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// Inclusive prefix sum over the 64 lanes of a wave.
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const uint32_t o = __shfl_up(v, off, kWave);
    if (lane >= off) v += o;
  }
  return v;
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

inline unsigned blocks_for(int64_t work, int threads) {
  return (unsigned)((work + threads - 1) / threads);
}

}  // namespace arc

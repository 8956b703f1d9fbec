// Shared device types and helpers for the gfx950 kernels of libhvd.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

namespace hvd {

constexpr int kWave = 64;

constexpr int kFragElems = 512;  // one 16x32 MFMA operand fragment: 64 lanes x 8 halves

// Round-to-nearest-even float -> bf16 bits (inputs are finite).
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// fp16 bits of v (round to nearest even) and back.
__device__ __forceinline__ uint16_t f2h(float v) { return __builtin_bit_cast(uint16_t, (_Float16)v); }
__device__ __forceinline__ float h2f(uint16_t b) { return (float)__builtin_bit_cast(_Float16, b); }

// Split v into hi + lo fp16 parts: hi = fp16(v), lo = fp16(v - hi).  hi + lo
// carries about 22 significant bits of v (fewer when lo is subnormal, where
// its absolute error is below 3e-8).
__device__ __forceinline__ void split_f16(float v, uint16_t& hi, uint16_t& lo) {
  hi = f2h(v);
  lo = f2h(v - h2f(hi));
}

// Offset (in halves) of element (row, col) inside a fragment-packed operand
// with `mtiles` 16-row tiles: fragment (kt = col/32, mt = row/16) is 64 lanes
// x 8 halves; lane = row%16 + 16*((col%32)/8), half = col%8.
__device__ __forceinline__ size_t afrag_off(int row, int col, int mtiles) {
  int kt = col >> 5, mt = row >> 4;
  int lane = (row & 15) + ((col & 31) >> 3) * 16;
  return ((size_t)(kt * mtiles + mt) * 64 + lane) * 8 + (col & 7);
}

__device__ __forceinline__ f32x4 mfma_f16(const u32x4& a, const u32x4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mfma_f16(const f16x8& a, const f16x8& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// Device-scope (write-through / coherent) stores and loads.  The L2 caches
// of the eight XCDs are not coherent with each other; data one workgroup
// hands to a workgroup of another XCD inside the same kernel goes through
// these (relaxed device-scope atomics: sc1 stores and loads, no cache-wide
// write-back or invalidate).  The writer waits for its stores (vmcnt(0))
// before it signals, and the reader loads only after seeing the signal.
__device__ __forceinline__ void store_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void store_dev_u32(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_dev(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_u32_dev(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u16_dev(uint16_t* p, uint16_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_u64_dev(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_u32_dev(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_u64_dev(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 16-byte device-scope loads and stores: raw buffer accesses with the sc1
// cache policy over a buffer that starts at `base` (wave-uniform) and is
// addressed by a byte offset below 2^31.
constexpr int kCachePolicySc1 = 16;
constexpr int kBufferWord3 = 0x00020000;  // raw buffer, 32-bit data format (gfx9)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, kBufferWord3);
}
__device__ __forceinline__ u32x4 ld_16_dev(const void* base, uint32_t byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(buf_rsrc(base), byte_off, 0, kCachePolicySc1);
}
__device__ __forceinline__ float4 ld_f4_dev(const void* base, uint32_t byte_off) {
  const u32x4 v = ld_16_dev(base, byte_off);
  return float4{__uint_as_float(v.x), __uint_as_float(v.y), __uint_as_float(v.z), __uint_as_float(v.w)};
}
__device__ __forceinline__ void st_16_dev(void* base, uint32_t byte_off, uint4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(u32x4{v.x, v.y, v.z, v.w}, buf_rsrc(base), byte_off, 0, kCachePolicySc1);
}
__device__ __forceinline__ void st_f4_dev(void* base, uint32_t byte_off, float4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z),
                                               __float_as_uint(v.w)},
                                         buf_rsrc(base), byte_off, 0, kCachePolicySc1);
}
// fp16 bits of (lo, hi) packed into one 32-bit word (lo in the low half)
__device__ __forceinline__ uint32_t pack_h2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) | ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
}

// Synchronisation points of work done inside a larger kernel (the one-launch
// verify step): wait() runs once the work's first constant inputs (weights,
// cached K/V) are requested and before any input another workgroup of the
// same kernel produces is read; done() runs after the work's outputs are
// written.  Stand-alone kernels use these no-ops.
struct NoHooks {
  static constexpr bool kDevOut = false;
  static constexpr int kPending = 0;
  __device__ __forceinline__ void wait() {}
  __device__ __forceinline__ void after_issue() {}
  __device__ __forceinline__ void done() {}
};

// s_waitcnt immediate that waits until at most n (< 64) vector memory
// operations are outstanding (lgkmcnt and expcnt left alone): vmcnt is
// split over bits 3:0 and 15:14.
__host__ __device__ constexpr int vmcnt_enc(int n) { return 0x0F70 | (n & 15) | ((n >> 4) << 14); }

// Across the four 16-lane rows of a wave: every lane gets the max (sum) of
// the values at its position l % 16 in all four rows.  The row-swap
// permutes of gfx950 do the xor-16 and xor-32 exchanges in the vector ALU,
// without the LDS round trip of a general shuffle; the pairs are combined
// in the same order as xor-16 then xor-32 shuffles would combine them.
__device__ __forceinline__ float rows_max(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows_sum(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

}  // namespace hvd

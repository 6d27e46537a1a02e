// Device-side helpers shared by the SKIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "skip.h"

namespace skip {

constexpr int kWave = 64;

typedef uint16_t bf16_t;   // raw bfloat16 bits
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // 16 bytes
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// ---- matrix cores (bf16 operands as 16-byte words, float32 accumulators)
// D (32 x 32) += A (32 x 16) . B (16 x 32): lane l holds A[l % 32][8(l / 32)
// .. +7], B[8(l / 32) .. +7][l % 32], and D[8(i / 4) + 4(l / 32) + i % 4][l % 32]
// in element i.
__device__ __forceinline__ f32x16_t mfma32_bf16(const u32x4& a, const u32x4& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}
// D (16 x 16) += A (16 x 32) . B (32 x 16): lane l holds A[l % 16][8(l / 16)
// .. +7], B[8(l / 16) .. +7][l % 16] and D[4(l / 16) .. +3][l % 16].
__device__ __forceinline__ f32x4_t mfma16_bf16(const u32x4& a, const u32x4& b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// ---- LDS staging
// Direct global->LDS load of 16 bytes per lane (global_load_lds_dwordx4):
// lane l's bytes land at LDS byte address lds + 16 * l (lds wave-uniform).
// Issued through inline assembly so that the compiler's wait-count pass does
// not treat it as a write that may alias every later LDS read (it would put a
// full vmcnt(0) before them); completion is awaited with wait_vmcnt.
__device__ __forceinline__ void lds_dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(lds)
               : "memory", "m0");
}
// LDS byte address of a shared-memory pointer, as a wave-uniform value.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p);
}
// Wait until at most N of this wave's vector-memory operations are pending
// (expcnt and lgkmcnt left unconstrained).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
  asm volatile("" ::: "memory");
}
// Workgroup barrier without a memory fence: the waves that write LDS wait for
// their own writes (vmcnt for direct loads, lgkmcnt for LDS stores) before it.
__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
// A wave-uniform 64-bit value moved to scalar registers.
__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ float bf16_to_f32(uint32_t h) {
  return __uint_as_float(h << 16);
}

// Round-to-nearest-even float -> bfloat16 (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// Two floats -> packed bf16 pair, round-to-nearest-even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// The eight bf16 values of a 16-byte word as floats (exact), in order.
__device__ __forceinline__ void unpack8_bf16(const u32x4& x, float* out) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    out[2 * w] = __uint_as_float(x[w] << 16);
    out[2 * w + 1] = __uint_as_float(x[w] & 0xffff0000u);
  }
}

// 16 bytes of T (4 floats or 8 bf16 values) as doubles (exact), in order.
template <typename T> struct Vec16;
template <> struct Vec16<float> { static constexpr int n = 4; };
template <> struct Vec16<bf16_t> { static constexpr int n = 8; };
template <typename T>
__device__ __forceinline__ void unpack16_f64(const u32x4& x, double* out);
template <>
__device__ __forceinline__ void unpack16_f64<float>(const u32x4& x, double* out) {
#pragma unroll
  for (int w = 0; w < 4; ++w) out[w] = (double)__uint_as_float(x[w]);
}
template <>
__device__ __forceinline__ void unpack16_f64<bf16_t>(const u32x4& x, double* out) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    out[2 * w] = (double)__uint_as_float(x[w] << 16);
    out[2 * w + 1] = (double)__uint_as_float(x[w] & 0xffff0000u);
  }
}

// Order-preserving map of a double onto uint64: a < b  <=>  key(a) < key(b),
// with -0.0 and +0.0 mapped to the same key.
__device__ __forceinline__ uint64_t order_key(double x) {
  uint64_t b = (x == 0.0) ? 0ull : (uint64_t)__double_as_longlong(x);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}

__device__ __forceinline__ int clampi(int v, int lo, int hi) {
  return v < lo ? lo : (v > hi ? hi : v);
}

// Offsets clamped into [0, total]; the pair is made non-decreasing.
__device__ __forceinline__ void range_of(const int32_t* off, int i, int total,
                                         int& a, int& b) {
  a = clampi(off[i], 0, total);
  b = clampi(off[i + 1], a, total);
}

// Publishing data to other workgroups of the same launch (a "last workgroup
// finishes" counter).  The L2 caches of the XCDs are not coherent with each
// other within a kernel, and an agent-scope fence writes back and invalidates
// the whole L2 of the XCD (costly for every other workgroup there).  Instead
// the shared values are written and read with agent-scope atomic accesses
// (coherent, sc1), each writer waits for its stores to be acknowledged before
// the workgroup barrier, and one thread then bumps the counter.
template <typename T>
__device__ __forceinline__ void store_shared(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T load_shared(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// every vector memory access of this wave (loads and stores) has completed
__device__ __forceinline__ void wait_all_vmem() {
  __builtin_amdgcn_s_waitcnt(0x0F70);            // vmcnt(0), expcnt and lgkmcnt untouched
}
// Called by every thread of the workgroup after its shared stores; returns
// true in every thread of the workgroup that completes `counter` to `total`.
__device__ __forceinline__ bool finish_and_check_last(int32_t* counter, int total, int* flag) {
  wait_all_vmem();
  __syncthreads();
  if (threadIdx.x == 0)
    *flag = (__hip_atomic_fetch_add(counter, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
             total - 1) ? 1 : 0;
  __syncthreads();
  return *flag != 0;
}

__device__ __forceinline__ double wave_sum_f64(double v) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) v += __shfl_xor(v, s, kWave);
  return v;
}

__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) v += __shfl_xor(v, s, kWave);
  return v;
}

__device__ __forceinline__ float wave_max_f32(float v) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) v = fmaxf(v, __shfl_xor(v, s, kWave));
  return v;
}

// Exclusive prefix sum of one uint32 per thread across the whole block, in
// thread order.  `sh` needs blockDim.x / 64 + 1 words.  Returns the exclusive
// prefix and writes the block total to *total.  Contains __syncthreads().
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t v, uint32_t* sh,
                                                         uint32_t* total) {
  const int lane = threadIdx.x & (kWave - 1);
  const int wid = threadIdx.x / kWave;
  const int nw = blockDim.x / kWave;
  uint32_t x = v;
#pragma unroll
  for (int s = 1; s < kWave; s <<= 1) {
    uint32_t y = __shfl_up(x, s, kWave);
    if (lane >= s) x += y;
  }
  if (lane == kWave - 1) sh[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int w = 0; w < nw; ++w) {
      uint32_t t = sh[w];
      sh[w] = run;
      run += t;
    }
    sh[nw] = run;
  }
  __syncthreads();
  uint32_t res = sh[wid] + x - v;
  *total = sh[nw];
  __syncthreads();
  return res;
}

}  // namespace skip

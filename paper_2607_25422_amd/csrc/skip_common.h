// Device-side helpers shared by the SKIP kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "skip.h"

namespace skip {

constexpr int kWave = 64;

typedef uint16_t bf16_t;   // raw bfloat16 bits
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));   // 16 bytes

__device__ __forceinline__ float bf16_to_f32(uint32_t h) {
  return __uint_as_float(h << 16);
}

// Round-to-nearest-even float -> bfloat16 (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
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

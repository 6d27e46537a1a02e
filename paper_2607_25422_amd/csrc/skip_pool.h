// Float64 means of row ranges of a [rows][d] matrix (internal to libskip.so):
// the mean-pooled question (paper Sec. 3.3, Def. B.2; Def. B.1 scoring
// vector) and the pooled passage keys (Def. B.3).
#pragma once

#include "skip_common.h"

namespace skip {

// Workgroup = (column slice of 64 lanes x kPoolChunks x 16 bytes, range);
// wave w sums rows w, w+4, ... (four rows, two 16-byte chunks each, in flight
// per lane); the four partial sums are combined in wave order through LDS.
// Questions are written as the scoring vector u = mean / sqrt(d) + w, passage
// keys as their mean.  The same workgroup body runs in the pooling launch and
// in the prune launch (passage keys beside the scoring).
constexpr int kPoolChunks = 2;

template <typename T>
struct PoolRanges {
  const T* src;
  const int32_t* offsets;
  int n;            // ranges
  int total;        // rows of src
  double* out;      // [n][d]
};

// Bytes of LDS one pooling workgroup uses (four waves' partial sums).
template <typename T>
constexpr size_t pool_lds_bytes() {
  return 4 * 64 * kPoolChunks * Vec16<T>::n * sizeof(double);
}

// One pooling workgroup (256 threads): range j of rg, column slice `slice`;
// `question` ranges are written as the scoring vector (mean / sqrt(d) + w).
// part: pool_lds_bytes<T>() of LDS.  Contains one __syncthreads().
template <typename T>
__device__ __forceinline__ void pool_block(const PoolRanges<T>& rg, int j, int slice,
                                           bool question, const T* __restrict__ w, int d,
                                           double* part) {
  constexpr int VEC = Vec16<T>::n;
  constexpr int CH = kPoolChunks;
  const T* __restrict__ src = rg.src;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int cc[CH];                            // first column of each chunk
  bool ok[CH];
#pragma unroll
  for (int h = 0; h < CH; ++h) {
    cc[h] = ((slice * CH + h) * 64 + lane) * VEC;
    ok[h] = cc[h] < d;
  }
  int t0, t1;
  range_of(rg.offsets, j, rg.total, t0, t1);
  double acc[CH][VEC];
#pragma unroll
  for (int h = 0; h < CH; ++h)
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[h][e] = 0.0;
  int t = t0 + wave;
  for (; t + 12 < t1; t += 16) {
    u32x4 x[4][CH];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int h = 0; h < CH; ++h)
        x[q][h] = ok[h] ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
                              src + (size_t)(t + 4 * q) * d + cc[h]))
                        : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int h = 0; h < CH; ++h) {
        double v[VEC];
        unpack16_f64<T>(x[q][h], v);
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[h][e] += v[e];
      }
  }
  for (; t < t1; t += 4) {
#pragma unroll
    for (int h = 0; h < CH; ++h) {
      if (!ok[h]) continue;
      u32x4 x = *reinterpret_cast<const u32x4*>(src + (size_t)t * d + cc[h]);
      double v[VEC];
      unpack16_f64<T>(x, v);
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[h][e] += v[e];
    }
  }
  // part[wave][lane][CH * VEC]
  double* mine = part + ((size_t)wave * 64 + lane) * (CH * VEC);
#pragma unroll
  for (int h = 0; h < CH; ++h)
#pragma unroll
    for (int e = 0; e < VEC; ++e) mine[h * VEC + e] = acc[h][e];
  __syncthreads();
  if (wave != 0) return;
  const int L = t1 - t0;
  const double rsd = 1.0 / sqrt((double)d);
  const size_t wstride = (size_t)64 * (CH * VEC);
#pragma unroll
  for (int h = 0; h < CH; ++h) {
    if (!ok[h]) continue;
    double wv[VEC];
    if (question && w) {
      unpack16_f64<T>(*reinterpret_cast<const u32x4*>(w + cc[h]), wv);
    } else {
#pragma unroll
      for (int e = 0; e < VEC; ++e) wv[e] = 0.0;
    }
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const int i = h * VEC + e;
      const double s = ((mine[i] + mine[wstride + i]) + mine[2 * wstride + i]) +
                       mine[3 * wstride + i];
      double m = (L > 0) ? s / (double)L : 0.0;
      if (question) m = m * rsd + wv[e];
      rg.out[(size_t)j * d + cc[h] + e] = m;
    }
  }
}

// One launch serves two independent sets of ranges: the questions (ranges
// 0..nq-1 of Qtok, written as the scoring vector) and the passages (the
// following ranges of Kh, written as their mean).  counters (or NULL): the
// per-question completion counters of the scoring launch, cleared here.
template <typename T>
__global__ void __launch_bounds__(256)
pool_kernel(PoolRanges<T> qr, const T* __restrict__ w, PoolRanges<T> pr, int d,
            int32_t* __restrict__ counters) {
  __shared__ double part[4 * 64 * kPoolChunks * Vec16<T>::n];
  const bool question = (int)blockIdx.y < qr.n;
  const int j = question ? (int)blockIdx.y : (int)blockIdx.y - qr.n;
  if (counters && question && blockIdx.x == 0 && threadIdx.x == 0) counters[j] = 0;
  pool_block<T>(question ? qr : pr, j, blockIdx.x, question, w, d, part);
}

// Questions (Qtok by q_offsets -> u, nq ranges) and passages (Kh by
// passage_offsets -> kbar, np ranges); either set may be empty.
inline hipError_t launch_pools(int dtype, int d, const void* Qtok, const int32_t* q_offsets,
                               int nq, int total_qtok, const void* w, double* u,
                               const void* Kh, const int32_t* passage_offsets, int np,
                               int total_tokens, double* kbar, hipStream_t s,
                               int32_t* counters = nullptr) {
  if (nq + np <= 0) return hipSuccess;
  if (dtype == SKIP_F32) {
    dim3 grid((d + 256 * kPoolChunks - 1) / (256 * kPoolChunks), nq + np);
    hipLaunchKernelGGL(pool_kernel<float>, grid, dim3(256), 0, s,
                       PoolRanges<float>{(const float*)Qtok, q_offsets, nq, total_qtok, u},
                       (const float*)w,
                       PoolRanges<float>{(const float*)Kh, passage_offsets, np, total_tokens,
                                         kbar},
                       d, counters);
  } else {
    dim3 grid((d + 512 * kPoolChunks - 1) / (512 * kPoolChunks), nq + np);
    hipLaunchKernelGGL(pool_kernel<bf16_t>, grid, dim3(256), 0, s,
                       PoolRanges<bf16_t>{(const bf16_t*)Qtok, q_offsets, nq, total_qtok, u},
                       (const bf16_t*)w,
                       PoolRanges<bf16_t>{(const bf16_t*)Kh, passage_offsets, np,
                                          total_tokens, kbar},
                       d, counters);
  }
  return hipGetLastError();
}

}  // namespace skip

// Stage 1 of the routing core: question-guided visual token pruning
// (paper App. B.1, Def. B.1; Alg. 1, scoring and TopK steps).
//
//   pool_question : u_b = mean(Q_b rows) / sqrt(d) + w          (float64,
//                   the row-range mean kernel shared with the passage keys)
//   score         : z_{b,i} = <u_b, V[b,i]>, s = sigmoid(z)     (float64 sums)
//   topk          : the k_b largest z of question b, lowest index on ties,
//                   written in ascending index order
//   gather        : V_kept rows = V[b, kept_idx]
//
// The score pass is the HBM stream of V: each wave streams rows with 16-byte
// loads (a full 1 KiB per wave instruction), several rows and several column
// chunks in flight per lane, against u_b staged once per workgroup in LDS.
#include "skip_common.h"
#include "skip_internal.h"
#include "skip_pool.h"
#include "skip_select.h"

namespace skip {

// ---------------------------------------------------------------------------
// Streaming GEMV in float64.  Workgroup = 4 waves = kScoreRows rows of one
// question; each wave handles kRowsPerWave rows, R at a time, U column chunks
// (of 64 lanes x 16 bytes) in flight per row.
constexpr int kScoreRows = 24;
constexpr int kScoreR = 6;
constexpr int kScoreU = 4;

template <typename T>
__global__ void __launch_bounds__(256)
score_kernel(const T* __restrict__ V, const double* __restrict__ u, int N, int d,
             double* __restrict__ z, float* __restrict__ scores) {
  constexpr int VEC = Vec16<T>::n;
  extern __shared__ double su[];          // [d]
  const int b = blockIdx.y;
  for (int c = threadIdx.x; c < d; c += blockDim.x) su[c] = u[(size_t)b * d + c];
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int rows_per_wave = kScoreRows / 4;
  const int r_begin = blockIdx.x * kScoreRows + wave * rows_per_wave;
  const int r_end = min(r_begin + rows_per_wave, N);
  const T* Vb = V + (size_t)b * N * d;

  for (int r0 = r_begin; r0 < r_end; r0 += kScoreR) {
    double acc[kScoreR];
#pragma unroll
    for (int rr = 0; rr < kScoreR; ++rr) acc[rr] = 0.0;
    for (int c0 = lane * VEC; c0 < d; c0 += 64 * VEC * kScoreU) {
      u32x4 x[kScoreR][kScoreU];
#pragma unroll
      for (int uu = 0; uu < kScoreU; ++uu) {
        const int c = c0 + uu * 64 * VEC;
#pragma unroll
        for (int rr = 0; rr < kScoreR; ++rr) {
          const int r = r0 + rr;
          if (c < d && r < r_end)
            x[rr][uu] = __builtin_nontemporal_load(
                reinterpret_cast<const u32x4*>(Vb + (size_t)r * d + c));
          else
            x[rr][uu] = u32x4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int uu = 0; uu < kScoreU; ++uu) {
        const int c = c0 + uu * 64 * VEC;
        if (c < d) {
          double w[VEC];
#pragma unroll
          for (int e = 0; e < VEC; ++e) w[e] = su[c + e];
#pragma unroll
          for (int rr = 0; rr < kScoreR; ++rr) {
            double v[VEC];
            unpack16_f64<T>(x[rr][uu], v);
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[rr] = fma(v[e], w[e], acc[rr]);
          }
        }
      }
    }
#pragma unroll
    for (int rr = 0; rr < kScoreR; ++rr) {
      const double t = wave_sum_f64(acc[rr]);
      const int r = r0 + rr;
      if (lane == 0 && r < r_end) {
        z[(size_t)b * N + r] = t;
        if (scores) scores[(size_t)b * N + r] = (float)(1.0 / (1.0 + exp(-t)));
      }
    }
  }
}

// ---------------------------------------------------------------------------
// One workgroup per question: exact top-k of the N logits.
constexpr int kSelThreads = 1024;
constexpr int kSelMaxPT = 16;     // N <= 16384

__global__ void __launch_bounds__(kSelThreads)
topk_kernel(const double* __restrict__ z, const int32_t* __restrict__ kept_offsets,
            int N, int total_kept, int32_t* __restrict__ kept_idx) {
  __shared__ SelectShared sh;
  __shared__ uint32_t scan_sh[20];
  const int b = blockIdx.x;
  int k0, k1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  const int kk = min(k1 - k0, N);
  const int C = (N + blockDim.x - 1) / blockDim.x;
  const int e0 = threadIdx.x * C;
  const int cnt = max(0, min(C, N - e0));
  uint64_t keys[kSelMaxPT];
#pragma unroll
  for (int j = 0; j < kSelMaxPT; ++j)
    keys[j] = (j < cnt) ? order_key(z[(size_t)b * N + e0 + j]) : 0ull;
  const uint32_t flags = block_select_top<kSelMaxPT>(keys, cnt, N, kk, &sh);
  uint32_t total;
  uint32_t pos = block_exclusive_scan(__popc(flags), scan_sh, &total);
#pragma unroll
  for (int j = 0; j < kSelMaxPT; ++j) {
    if (flags & (1u << j)) {
      if (pos < (uint32_t)kk) kept_idx[k0 + pos] = e0 + j;
      ++pos;
    }
  }
}

// ---------------------------------------------------------------------------
// V_kept[r] = V[b][kept_idx[r]].  A workgroup stages the indices of its
// kGatherRows rows in LDS, then each wave copies rows with 16-byte accesses.
constexpr int kGatherRows = 16;

template <typename T>
__global__ void __launch_bounds__(256)
gather_kernel(const T* __restrict__ V, const int32_t* __restrict__ kept_offsets,
              const int32_t* __restrict__ kept_idx, int N, int d, int total_kept,
              T* __restrict__ V_kept) {
  constexpr int VEC = Vec16<T>::n;
  __shared__ int32_t src[kGatherRows];
  const int b = blockIdx.y;
  int k0, k1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  const int i0 = blockIdx.x * kGatherRows;
  if (threadIdx.x < kGatherRows) {
    const int i = i0 + threadIdx.x;
    src[threadIdx.x] = (k0 + i < k1) ? clampi(kept_idx[k0 + i], 0, N - 1) : -1;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int rr = wave; rr < kGatherRows; rr += 4) {
    const int s = src[rr];
    if (s < 0) continue;
    const T* from = V + ((size_t)b * N + s) * d;
    T* to = V_kept + (size_t)(k0 + i0 + rr) * d;
    for (int c = lane * VEC; c < d; c += 64 * VEC)
      *reinterpret_cast<u32x4*>(to + c) = *reinterpret_cast<const u32x4*>(from + c);
  }
}

// ---------------------------------------------------------------------------
// Launchers.
hipError_t launch_pool_question(const skip_problem_t& p, const void* Qtok,
                                const int32_t* q_offsets, const void* w_bias,
                                double* u, hipStream_t s) {
  return launch_pools(p.dtype, p.d, Qtok, q_offsets, p.B, p.total_qtok, w_bias, u, nullptr,
                      nullptr, 0, 0, nullptr, s);
}

hipError_t launch_score(const skip_problem_t& p, const void* V, const double* u,
                        double* z, float* scores, hipStream_t s) {
  dim3 grid((p.N + kScoreRows - 1) / kScoreRows, p.B);
  const size_t lds = (size_t)p.d * sizeof(double);
  if (p.dtype == SKIP_F32)
    hipLaunchKernelGGL(score_kernel<float>, grid, dim3(256), lds, s,
                       (const float*)V, u, p.N, p.d, z, scores);
  else
    hipLaunchKernelGGL(score_kernel<bf16_t>, grid, dim3(256), lds, s,
                       (const bf16_t*)V, u, p.N, p.d, z, scores);
  return hipGetLastError();
}

hipError_t launch_topk(const skip_problem_t& p, const double* z,
                       const int32_t* kept_offsets, int32_t* kept_idx, hipStream_t s) {
  hipLaunchKernelGGL(topk_kernel, dim3(p.B), dim3(kSelThreads), 0, s, z, kept_offsets,
                     p.N, p.total_kept, kept_idx);
  return hipGetLastError();
}

hipError_t launch_gather(const skip_problem_t& p, const void* V,
                         const int32_t* kept_offsets, const int32_t* kept_idx,
                         void* V_kept, hipStream_t s) {
  if (p.k_max <= 0) return hipSuccess;
  dim3 grid((p.k_max + kGatherRows - 1) / kGatherRows, p.B);
  if (p.dtype == SKIP_F32)
    hipLaunchKernelGGL(gather_kernel<float>, grid, dim3(256), 0, s, (const float*)V,
                       kept_offsets, kept_idx, p.N, p.d, p.total_kept, (float*)V_kept);
  else
    hipLaunchKernelGGL(gather_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)V,
                       kept_offsets, kept_idx, p.N, p.d, p.total_kept, (bf16_t*)V_kept);
  return hipGetLastError();
}

}  // namespace skip

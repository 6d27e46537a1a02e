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
#include <algorithm>
#include <type_traits>

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

// Rows [24 rb, 24 rb + 24) of question b: z = <u_b, v_i> in float64 (and
// sigma(z) if asked).  su: u_b in LDS (d doubles, filled here).  z is
// written with device-coherent stores: the question's top-k may run on
// another XCD.
template <typename T>
__device__ __forceinline__ void score_rows(const T* __restrict__ V, const double* __restrict__ u,
                                           int N, int d, int b, int rb, double* __restrict__ z,
                                           float* __restrict__ scores, double* su) {
  constexpr int VEC = Vec16<T>::n;
  for (int c = threadIdx.x; c < d; c += blockDim.x) su[c] = u[(size_t)b * d + c];
  __syncthreads();

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int rows_per_wave = kScoreRows / 4;
  const int r_begin = rb * kScoreRows + wave * rows_per_wave;
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
        store_shared(&z[(size_t)b * N + r], t);
        if (scores) scores[(size_t)b * N + r] = (float)(1.0 / (1.0 + exp(-t)));
      }
    }
  }
}

// Exact top-k of question b's N logits by one workgroup (any size); the
// logits are read device-coherently.  sh: LDS for the selection; scan_sh:
// blockDim.x / 64 + 1 words.  Kept indices ascending.
template <int MAXPT>
__device__ __forceinline__ void topk_block(const double* __restrict__ z, int b, int N,
                                           const int32_t* __restrict__ kept_offsets,
                                           int total_kept, int32_t* __restrict__ kept_idx,
                                           SelectShared* sh, uint32_t* scan_sh) {
  int k0, k1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  const int kk = min(k1 - k0, N);
  const int C = (N + blockDim.x - 1) / blockDim.x;
  const int e0 = threadIdx.x * C;
  const int cnt = max(0, min(C, N - e0));
  uint64_t keys[MAXPT];
#pragma unroll
  for (int j = 0; j < MAXPT; ++j)
    keys[j] = (j < cnt) ? order_key(load_shared(&z[(size_t)b * N + e0 + j])) : 0ull;
  const SelectMask<MAXPT> flags = block_select_top<MAXPT>(keys, cnt, N, kk, sh);
  uint32_t total;
  uint32_t pos = block_exclusive_scan((uint32_t)__popcll((uint64_t)flags), scan_sh, &total);
#pragma unroll
  for (int j = 0; j < MAXPT; ++j) {
    if (flags & ((SelectMask<MAXPT>)1 << j)) {
      if (pos < (uint32_t)kk) kept_idx[k0 + pos] = e0 + j;
      ++pos;
    }
  }
}

// The prune stage in one launch: RB = ceil(N / kScoreRows) scoring
// workgroups per question, question-major, then (optionally) the pooling
// workgroups of the passage keys.  The last scoring workgroup of a question
// to finish (a per-question counter, cleared by the question pooling before
// the launch and again here after use) selects the question's top k, so the
// top-k runs beside the scoring of later questions and the key pooling
// instead of as a launch of its own.
template <typename T, int MAXPT>
__global__ void __launch_bounds__(256, 3)   // three waves per SIMD for the scoring stream
prune_kernel(const T* __restrict__ V, const double* __restrict__ u, int N, int d, int B,
             int RB, double* __restrict__ z, float* __restrict__ scores,
             const int32_t* __restrict__ kept_offsets, int total_kept,
             int32_t* __restrict__ kept_idx, int32_t* __restrict__ counters,
             PoolRanges<T> keys, int key_slices) {
  extern __shared__ __align__(16) double lds[];
  __shared__ int last;
  const int bid = blockIdx.x;
  const int n_score = RB * B;
  if (bid >= n_score) {
    const int kb = bid - n_score;
    pool_block<T>(keys, kb / key_slices, kb % key_slices, false, nullptr, d, lds);
    return;
  }
  const int b = bid / RB, rb = bid % RB;
  score_rows<T>(V, u, N, d, b, rb, z, scores, lds);
  if (!finish_and_check_last(&counters[b], RB, &last)) return;
  SelectShared* sh = reinterpret_cast<SelectShared*>(lds);
  uint32_t* scan_sh = reinterpret_cast<uint32_t*>(sh + 1);
  topk_block<MAXPT>(z, b, N, kept_offsets, total_kept, kept_idx, sh, scan_sh);
  if (threadIdx.x == 0) store_shared(&counters[b], 0);
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
  const uint32_t flags = block_select_top_wide<kSelMaxPT>(keys, cnt, N, kk, &sh);
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
                                double* u, int32_t* counters, hipStream_t s) {
  return launch_pools(p.dtype, p.d, Qtok, q_offsets, p.B, p.total_qtok, w_bias, u, nullptr,
                      nullptr, 0, 0, nullptr, s, counters);
}

hipError_t launch_prune(const skip_problem_t& p, const void* V, const double* u, double* z,
                        float* scores, const int32_t* kept_offsets, int32_t* kept_idx,
                        int32_t* counters, const void* Kh, const int32_t* passage_offsets,
                        int n_keys, double* kbar, hipStream_t s) {
  if (p.B <= 0 || p.N <= 0) return hipSuccess;
  const int RB = (p.N + kScoreRows - 1) / kScoreRows;
  const int C = (p.N + 255) / 256;              // logits per thread in the top-k
  if (C > 64) return hipErrorInvalidValue;
  auto go = [&](auto tag, auto maxpt) -> hipError_t {
    using T = decltype(tag);
    constexpr int MAXPT = decltype(maxpt)::value;
    const int slices = (p.d + 64 * kPoolChunks * Vec16<T>::n - 1) / (64 * kPoolChunks * Vec16<T>::n);
    const size_t lds = std::max({(size_t)p.d * sizeof(double), pool_lds_bytes<T>(),
                                 sizeof(SelectShared) + 20 * sizeof(uint32_t)});
    const long long grid = (long long)RB * p.B + (long long)slices * n_keys;
    if (grid > INT32_MAX) return hipErrorInvalidValue;
    hipLaunchKernelGGL((prune_kernel<T, MAXPT>), dim3((unsigned)grid), dim3(256), lds, s,
                       (const T*)V, u, p.N, p.d, p.B, RB, z, scores, kept_offsets,
                       p.total_kept, kept_idx, counters,
                       PoolRanges<T>{(const T*)Kh, passage_offsets, n_keys, p.total_tokens, kbar},
                       slices);
    return hipGetLastError();
  };
  auto by_pt = [&](auto tag) -> hipError_t {
    if (C <= 16) return go(tag, std::integral_constant<int, 16>{});
    if (C <= 32) return go(tag, std::integral_constant<int, 32>{});
    return go(tag, std::integral_constant<int, 64>{});
  };
  if (p.dtype == SKIP_F32) return by_pt(float{});
  return by_pt(bf16_t{});
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

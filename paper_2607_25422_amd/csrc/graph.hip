// Bipartite graph between kept visual tokens and retrieved passages
// (paper App. B.3, Def. B.3 edge rule; Alg. 1, graph step).
//
//   passage_keys : kbar_j = mean over the tokens of passage j of Kh[m] (all
//                  heads flattened), float64 sums
//   edge_dot     : float64 partial sums of <q_i, kbar_j>, |q_i|^2, |kbar_j|^2
//                  over slices of d
//   (cosine)       c_ij = <q_i, kbar_j> / (|q_i| |kbar_j|), 0 when a norm is 0,
//                  formed from the partial sums by the selection kernel
//   edge_select  : per question, the E_b = min(ceil(avg_degree * k_b),
//                  k_b * P_b) largest cosines (lower flattened index i*P_b+j
//                  on ties) -> one 64-bit neighbour mask per kept row, and
//                  optionally the graph in CSR form.  Also selectable: the
//                  scaled dot product of eq. (bsca) instead of the cosine,
//                  the top-beta fraction of the pairs (Sec. 3.5) or a
//                  per-row cut instead of the per-question budget
//   csr_to_mask  : neighbour masks from a caller-given CSR graph
#include "skip_common.h"
#include "skip_internal.h"
#include "skip_pool.h"
#include "skip_select.h"

namespace skip {

template <typename T> __device__ __forceinline__ float elem_f32(const T* p, size_t i);
template <> __device__ __forceinline__ float elem_f32<float>(const float* p, size_t i) {
  return p[i];
}
template <> __device__ __forceinline__ float elem_f32<bf16_t>(const bf16_t* p, size_t i) {
  return bf16_to_f32(p[i]);
}

// ---------------------------------------------------------------------------
// Edge dot products on the float64 matrix cores, split over d.
// Workgroup = (512-column slice, 64 kept rows x 16 passages, question); wave w
// owns rows 16w..16w+15 of the block.  v_mfma_f64_16x16x4_f64 takes one
// element of A (rows x 4 columns) and one of B (4 columns x passages) per
// lane: lane l supplies row/passage l % 16 and column slot l / 16.  The
// contraction order over columns is free, so column slot kk of MFMA m (m =
// 0..7 within a 32-column step) is column 8*kk + m: every lane then reads 8
// consecutive columns of its row (one 16-byte load) and of its passage key,
// straight from global memory.  Each lane also sums the squares of the values
// it loads (partial row and key norms).  Results per slice are summed in
// slice order by the selection kernel.
constexpr int kEdRows = 64;
constexpr int kEdPT = 16;
constexpr int kEdSlice = 512;
constexpr int kEdSteps = 4;

typedef double f64x4_t __attribute__((ext_vector_type(4)));

template <typename T>
__device__ __forceinline__ void load8_f64(const T* p, bool ok, double* out);
template <>
__device__ __forceinline__ void load8_f64<bf16_t>(const bf16_t* p, bool ok, double* out) {
  u32x4 x = ok ? *reinterpret_cast<const u32x4*>(p) : u32x4{0u, 0u, 0u, 0u};
  unpack_f64<bf16_t>(x, out);
}
template <>
__device__ __forceinline__ void load8_f64<float>(const float* p, bool ok, double* out) {
  u32x4 x0 = ok ? *reinterpret_cast<const u32x4*>(p) : u32x4{0u, 0u, 0u, 0u};
  u32x4 x1 = ok ? *reinterpret_cast<const u32x4*>(p + 4) : u32x4{0u, 0u, 0u, 0u};
  unpack_f64<float>(x0, out);
  unpack_f64<float>(x1, out + 4);
}

template <typename T>
__global__ void __launch_bounds__(256)
edge_dot_kernel(const T* __restrict__ qbase, const int32_t* __restrict__ kept_idx, int N,
                const int32_t* __restrict__ kept_offsets,
                const int32_t* __restrict__ query_passages, const double* __restrict__ kbar,
                const float* __restrict__ pkeys, int d, int total_kept, int total_passages,
                int k_max, int P_max, int S, int n_pt, double* __restrict__ part,
                double* __restrict__ qn2p, double* __restrict__ kn2p) {
  const int s = blockIdx.x, b = blockIdx.z;
  const int rb = blockIdx.y / n_pt, pt = blockIdx.y % n_pt;
  int k0, k1, p0, p1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  range_of(query_passages, b, total_passages, p0, p1);
  const int kq = min(k1 - k0, k_max);
  const int P = min(min(p1 - p0, P_max), 64);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rt0 = rb * kEdRows + wave * 16;          // first row of this wave
  if (rt0 >= kq || pt * kEdPT >= P) return;          // whole wave (no barriers)
  const int c_begin = s * kEdSlice, c_end = min(d, c_begin + kEdSlice);
  const int l16 = lane & 15, kk = lane >> 4;
  const int row = rt0 + l16, pj = pt * kEdPT + l16;
  const bool row_ok = row < kq, key_ok = pj < P;
  const T* qrow = qbase;          // never read unless row_ok
  if (row_ok) {
    if (kept_idx) {
      const int src = clampi(kept_idx[k0 + row], 0, N - 1);
      qrow = qbase + ((size_t)b * N + src) * d;
    } else {
      qrow = qbase + (size_t)(k0 + row) * d;
    }
  }
  const size_t krow = (size_t)(p0 + (key_ok ? pj : 0)) * d;

  f64x4_t acc = {0.0, 0.0, 0.0, 0.0};
  double qq = 0.0, k2 = 0.0;
  // kEdSteps 32-column steps per iteration: every load of the iteration is
  // issued before the first product, so each wave waits once per 128 columns.
  for (int c0 = c_begin; c0 < c_end; c0 += 32 * kEdSteps) {
    double qa[kEdSteps][8], kv[kEdSteps][8];
#pragma unroll
    for (int st = 0; st < kEdSteps; ++st) {
      const int c = c0 + 32 * st + 8 * kk;
      const bool in = c < c_end;               // d is a multiple of 8
      load8_f64<T>(qrow + c, row_ok && in, qa[st]);
      if (pkeys) {
        load8_f64<float>(pkeys + krow + c, key_ok && in, kv[st]);
      } else if (key_ok && in) {
        const double2* kp = reinterpret_cast<const double2*>(kbar + krow + c);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const double2 t = kp[q];
          kv[st][2 * q] = t.x;
          kv[st][2 * q + 1] = t.y;
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) kv[st][e] = 0.0;
      }
    }
#pragma unroll
    for (int st = 0; st < kEdSteps; ++st)
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        acc = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[st][m], kv[st][m], acc, 0, 0, 0);
        qq = fma(qa[st][m], qa[st][m], qq);
        k2 = fma(kv[st][m], kv[st][m], k2);
      }
  }
  // lanes l16, l16+16, l16+32, l16+48 hold the four column slots of one row/key
  qq += __shfl_xor(qq, 16, 64);
  qq += __shfl_xor(qq, 32, 64);
  k2 += __shfl_xor(k2, 16, 64);
  k2 += __shfl_xor(k2, 32, 64);
  const size_t base = (size_t)b * S + s;
  // D[i][j]: register r of lane l holds row 4*r + l/16, passage column l % 16
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int i = rt0 + 4 * r + kk;
    if (i < kq && key_ok) part[(base * k_max + i) * P_max + pj] = acc[r];
  }
  if (kk == 0) {
    if (pt == 0 && row_ok) qn2p[base * k_max + row] = qq;
    if (rb == 0 && wave == 0 && key_ok) kn2p[base * P_max + pj] = k2;
  }
}

// ---------------------------------------------------------------------------
// Edge selection, one workgroup per question.
constexpr int kGSelThreads = 1024;
constexpr int kGSelMaxPT = 16;     // k_b * P_b <= 16384

// Edges a question keeps under each cut (the same arithmetic on every side).
__device__ __forceinline__ long long edges_of_question(int k, int P, int rule,
                                                       double avg_degree, double beta) {
  const long long n = min((long long)k * P, (long long)kGSelThreads * kGSelMaxPT);
  if (rule == SKIP_EDGE_ROW_TOP)
    return (long long)k * (long long)fmin((double)P, ceil(avg_degree));
  const double want = (rule == SKIP_EDGE_TOP_FRACTION) ? ceil(beta * (double)n - 1e-9)
                                                       : ceil(avg_degree * (double)k);
  return (long long)fmin((double)n, fmax(0.0, want));
}

__global__ void __launch_bounds__(kGSelThreads)
edge_select_kernel(const double* __restrict__ part, const double* __restrict__ qn2p,
                   const double* __restrict__ kn2p, int S,
                   const int32_t* __restrict__ kept_offsets,
                   const int32_t* __restrict__ query_passages, int B, int total_kept,
                   int total_passages, int k_max, int P_max, int d, double avg_degree,
                   int rule, int metric, double beta, const uint8_t* __restrict__ keep,
                   uint64_t* __restrict__ rowmask, int32_t* __restrict__ rowptr_out,
                   int32_t* __restrict__ col_out) {
  __shared__ SelectShared sh;
  __shared__ uint32_t scan_sh[20];
  __shared__ uint8_t flag[kGSelThreads * kGSelMaxPT];
  __shared__ uint64_t rkeys[kGSelThreads * kGSelMaxPT];   // per-row cut only
  const int b = blockIdx.x;
  int k0, k1, p0, p1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  range_of(query_passages, b, total_passages, p0, p1);
  const int k = min(k1 - k0, k_max);
  const int P = min(min(p1 - p0, P_max), 64);
  const int n = min(k * P, kGSelThreads * kGSelMaxPT);
  // passages the verification gate dropped take no edge and do not count in
  // the budget: their candidates get the lowest key
  uint64_t pkeep = (P >= 64) ? ~0ull : ((1ull << P) - 1ull);
  if (keep) {
    pkeep = 0ull;
    for (int j = 0; j < P; ++j) pkeep |= (keep[p0 + j] ? 1ull : 0ull) << j;
  }
  const int Pk = __popcll(pkeep);
  const int E = (int)edges_of_question(k, Pk, rule, avg_degree, beta);
  const double inv_sqrt_d = 1.0 / sqrt((double)d);

  const int C = (n + blockDim.x - 1) / blockDim.x;
  const int e0 = threadIdx.x * C;
  const int cnt = max(0, min(C, n - e0));
  // compatibility of (i, j) from the per-slice partial sums, in slice order
  uint64_t keys[kGSelMaxPT];
#pragma unroll
  for (int jj = 0; jj < kGSelMaxPT; ++jj) {
    keys[jj] = 0ull;
    if (jj < cnt) {
      const int f = e0 + jj, i = f / P, j = f % P;
      double dot = 0.0, q2 = 0.0, k2 = 0.0;
      for (int sl0 = 0; sl0 < S; sl0 += 8) {
        double pd[8], pq[8], pk[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const size_t base = (size_t)b * S + min(sl0 + u, S - 1);
          pd[u] = part[(base * k_max + i) * P_max + j];
          pq[u] = qn2p[base * k_max + i];
          pk[u] = kn2p[base * P_max + j];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u)
          if (sl0 + u < S) { dot += pd[u]; q2 += pq[u]; k2 += pk[u]; }
      }
      double c;
      if (metric == SKIP_EDGE_DOT) {
        c = dot * inv_sqrt_d;
      } else {
        const double nq = sqrt(q2), nk = sqrt(k2);
        c = (nq > 0.0 && nk > 0.0) ? dot / (nq * nk) : 0.0;
      }
      keys[jj] = ((pkeep >> j) & 1ull) ? order_key(c) : 0ull;
    }
  }
  uint32_t flags;
  if (rule == SKIP_EDGE_ROW_TOP) {
    // every row keeps its D largest (lower passage first on ties)
#pragma unroll
    for (int jj = 0; jj < kGSelMaxPT; ++jj)
      if (jj < cnt) rkeys[e0 + jj] = keys[jj];
    __syncthreads();
    const int D = (int)fmin((double)Pk, ceil(avg_degree));
    for (int i = threadIdx.x; i < k && (i + 1) * P <= n; i += blockDim.x) {
      const uint64_t* rk = rkeys + i * P;
      for (int j = 0; j < P; ++j) {
        const uint64_t kj = rk[j];
        int rank = 0;
        for (int t = 0; t < P; ++t) {
          const uint64_t kt = rk[t];
          rank += (kt > kj || (kt == kj && t < j)) ? 1 : 0;
        }
        flag[i * P + j] = rank < D ? 1u : 0u;
      }
    }
    __syncthreads();
    flags = 0u;
#pragma unroll
    for (int jj = 0; jj < kGSelMaxPT; ++jj)
      if (jj < cnt && flag[e0 + jj]) flags |= 1u << jj;
  } else {
    flags = block_select_top<kGSelMaxPT>(keys, cnt, n, E, &sh);
#pragma unroll
    for (int j = 0; j < kGSelMaxPT; ++j)
      if (j < cnt) flag[e0 + j] = (flags >> j) & 1u;
    __syncthreads();
  }
  for (int i = threadIdx.x; i < k; i += blockDim.x) {
    uint64_t m = 0;
    if (P > 0 && (i + 1) * P <= n)
      for (int j = 0; j < P; ++j) m |= (uint64_t)flag[i * P + j] << j;
    rowmask[k0 + i] = m;
  }
  if (rowptr_out == nullptr || col_out == nullptr) return;

  // CSR: the edges of question b start after those of questions 0..b-1.
  long long base = 0;
  for (int bb = 0; bb < b; ++bb) {
    int a0, a1, q0, q1;
    range_of(kept_offsets, bb, total_kept, a0, a1);
    range_of(query_passages, bb, total_passages, q0, q1);
    const int kq = min(a1 - a0, k_max), Pq = min(min(q1 - q0, P_max), 64);
    int Pkq = Pq;
    if (keep) {
      Pkq = 0;
      for (int j = 0; j < Pq; ++j) Pkq += keep[q0 + j] ? 1 : 0;
    }
    base += edges_of_question(kq, Pkq, rule, avg_degree, beta);
  }
  uint32_t total;
  uint32_t pos = block_exclusive_scan(__popc(flags), scan_sh, &total);
  const long long cap = (long long)total_kept * P_max;
#pragma unroll
  for (int j = 0; j < kGSelMaxPT; ++j) {
    if (j < cnt) {
      const int f = e0 + j;
      if (P > 0 && f % P == 0) {
        const int i = f / P;
        if (i < k) rowptr_out[k0 + i] = (int32_t)(base + pos);
      }
      if (flags & (1u << j)) {
        if (base + pos < cap) col_out[base + pos] = f % P;
        ++pos;
      }
    }
  }
  // Rows beyond the candidate range (P == 0): they have no edges.
  if (P == 0)
    for (int i = threadIdx.x; i < k; i += blockDim.x) rowptr_out[k0 + i] = (int32_t)base;
  if (b == B - 1 && threadIdx.x == 0) rowptr_out[total_kept] = (int32_t)(base + total);
}

// ---------------------------------------------------------------------------
// Neighbour masks from a caller-given CSR graph.
__global__ void __launch_bounds__(256)
csr_to_mask_kernel(const int32_t* __restrict__ kept_offsets,
                   const int32_t* __restrict__ query_passages,
                   const int32_t* __restrict__ rowptr, const int32_t* __restrict__ col,
                   int total_kept, int total_passages, int total_edges,
                   uint64_t* __restrict__ rowmask) {
  const int b = blockIdx.y;
  int k0, k1, p0, p1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  range_of(query_passages, b, total_passages, p0, p1);
  const int P = min(p1 - p0, 64);
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (k0 + i >= k1) return;
  int e0, e1;
  range_of(rowptr, k0 + i, total_edges, e0, e1);
  uint64_t m = 0;
  for (int e = e0; e < e1; ++e) {
    const int j = col[e];
    if (j >= 0 && j < P) m |= 1ull << j;
  }
  rowmask[k0 + i] = m;
}

// ---------------------------------------------------------------------------
hipError_t launch_passage_keys(const skip_problem_t& p, const void* Kh,
                               const int32_t* passage_offsets, double* kbar,
                               hipStream_t s) {
  if (p.total_passages <= 0) return hipSuccess;
  return launch_pools(p.dtype, p.d, nullptr, nullptr, 0, 0, nullptr, nullptr, Kh,
                      passage_offsets, p.total_passages, p.total_tokens, kbar, s);
}

int edge_slices(const skip_problem_t& p) { return (p.d + kEdSlice - 1) / kEdSlice; }

hipError_t launch_edge_dot(const skip_problem_t& p, QuerySource q,
                           const int32_t* kept_offsets, const int32_t* query_passages,
                           const double* kbar, const float* passage_keys, EdgePartials ep,
                           hipStream_t s) {
  if (p.k_max <= 0 || p.P_max <= 0) return hipSuccess;
  const int S = edge_slices(p);
  const int n_pt = (p.P_max + kEdPT - 1) / kEdPT;
  dim3 grid(S, ((p.k_max + kEdRows - 1) / kEdRows) * n_pt, p.B);
  if (p.dtype == SKIP_F32)
    hipLaunchKernelGGL(edge_dot_kernel<float>, grid, dim3(256), 0, s,
                       (const float*)q.base, q.kept_idx, q.N, kept_offsets, query_passages,
                       kbar, passage_keys, p.d, p.total_kept, p.total_passages, p.k_max,
                       p.P_max, S, n_pt, ep.part, ep.qn2, ep.kn2);
  else
    hipLaunchKernelGGL(edge_dot_kernel<bf16_t>, grid, dim3(256), 0, s,
                       (const bf16_t*)q.base, q.kept_idx, q.N, kept_offsets,
                       query_passages, kbar, passage_keys, p.d, p.total_kept,
                       p.total_passages, p.k_max, p.P_max, S, n_pt, ep.part, ep.qn2, ep.kn2);
  return hipGetLastError();
}

hipError_t launch_edge_select(const skip_problem_t& p, EdgePartials ep,
                              const int32_t* kept_offsets, const int32_t* query_passages,
                              uint64_t* rowmask, int32_t* rowptr_out, int32_t* col_out,
                              hipStream_t s, const uint8_t* passage_keep) {
  hipLaunchKernelGGL(edge_select_kernel, dim3(p.B), dim3(kGSelThreads), 0, s, ep.part,
                     ep.qn2, ep.kn2, edge_slices(p), kept_offsets, query_passages, p.B,
                     p.total_kept, p.total_passages, p.k_max, p.P_max, p.d, p.avg_degree,
                     p.edge_rule, p.edge_metric, p.edge_beta, passage_keep, rowmask,
                     rowptr_out, col_out);
  return hipGetLastError();
}

hipError_t launch_csr_to_mask(const skip_problem_t& p, const int32_t* kept_offsets,
                              const int32_t* query_passages, const int32_t* edge_rowptr,
                              const int32_t* edge_col, uint64_t* rowmask, hipStream_t s) {
  if (p.k_max <= 0) return hipSuccess;
  dim3 grid((p.k_max + 255) / 256, p.B);
  hipLaunchKernelGGL(csr_to_mask_kernel, grid, dim3(256), 0, s, kept_offsets,
                     query_passages, edge_rowptr, edge_col, p.total_kept,
                     p.total_passages, p.total_edges, rowmask);
  return hipGetLastError();
}

}  // namespace skip

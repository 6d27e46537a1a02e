// Bipartite graph between kept visual tokens and retrieved passages
// (paper App. B.3, Def. B.3 edge rule; Alg. 1, graph step).
//
//   passage_keys : kbar_j = mean over the tokens of passage j of Kh[m] (all
//                  heads flattened), float64 sums
//   edge_dot     : float64 partial sums of <q_i, kbar_j>, |q_i|^2, |kbar_j|^2
//                  over slices of d
//   edge_keys    : c_ij = <q_i, kbar_j> / (|q_i| |kbar_j|) (0 when a norm is
//                  0) from the partial sums in slice order, as an
//                  order-preserving 64-bit key per candidate
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
#include "skip_plan.h"
#include "skip_pool.h"
#include "skip_select.h"

namespace skip {

// ---------------------------------------------------------------------------
// Edge dot products on the float64 matrix cores, split over d.
// Workgroup = (question, 256-column slice, block of 64 kept rows); the slices
// and row blocks of a question run on one XCD (workgroup id L goes to XCD
// L % 8), where they share the keys in the L2.  v_mfma_f64_16x16x4_f64 takes
// one element of A (16 rows x 4 columns) and one of B (4 columns x 16
// passages) per lane: lane l supplies row/passage l % 16 and column slot
// l / 16.  The contraction order over columns is free, so column slot kk of
// MFMA m within a group of 4·E columns (E = 8 bf16 or 4 f32 per 16-byte
// chunk) is column E*kk + m: a lane then reads one 16-byte chunk of its row
// and E consecutive key values per group.
//   * Wave w takes the 16-row tile w of the block and reads its rows' slice
//     straight from memory, one 16-byte chunk per lane and group (bf16: all
//     chunks loaded into registers before the keys are staged; f32, twice
//     the chunks: each where it is used).
//   * The passage keys of the slice sit in LDS as float64, 16 passages at a
//     time, read by all four waves (float64 keys by direct global->LDS loads
//     issued before the rows).  With only the keys in LDS (33 KiB), three
//     bf16 workgroups share a CU (registers allow three waves per SIMD), so
//     one wave's loads and conversions overlap another's matrix products.
// Each lane also sums the squares of its row values (partial row norms); the
// key norms come from the keys in LDS (row block 0).  Results per slice are
// summed in slice order by the key launch.
constexpr int kEdCols = 256;               // columns per slice
constexpr int kEdRows = 64;                // rows per workgroup (a 16-row tile per wave)
constexpr int kEdPT = 16;                  // passages per tile
constexpr int kEdKeyStride = kEdCols + 2;  // doubles per key row in LDS (bank spread)

typedef double f64x4_t __attribute__((ext_vector_type(4)));

struct EdgeDotArgs {
  const int32_t* kept_idx;     // NULL: rows are [total_kept][d]; else V [B][N][d]
  int N;
  const int32_t* kept_offsets;
  const int32_t* query_passages;
  const double* kbar;          // [total_passages][d] float64 keys, or
  const float* pkeys;          // [total_passages][d] caller-given keys
  int d, total_kept, total_passages, k_max, P_max, B, S, RB;
  double* part;                // [B][S][k_max][P_max] partial <q_i, k̄_j>
  double* qn2p;                // [B][S][k_max]        partial |q_i|^2
  double* kn2p;                // [B][S][P_max]        partial |k̄_j|^2
};

template <typename T>
__global__ void __launch_bounds__(256, sizeof(T) == 2 ? 3 : 2)   // waves per SIMD
edge_dot_kernel(const T* __restrict__ rows, EdgeDotArgs a) {
  constexpr int E = 16 / (int)sizeof(T);          // columns per 16-byte chunk
  constexpr int NG = kEdCols / (4 * E);            // groups of 4·E columns per slice
  __shared__ __align__(16) double ks[kEdPT * kEdKeyStride];
  const int L = blockIdx.x, xcd = L & 7, jl = L >> 3;
  const int per_q = a.S * a.RB;
  const int b = xcd + 8 * (jl / per_q);
  const int s = (jl % per_q) % a.S, rb = (jl % per_q) / a.S, tid = threadIdx.x;
  if (b >= a.B) return;
  int k0, k1, p0, p1;
  range_of(a.kept_offsets, b, a.total_kept, k0, k1);
  range_of(a.query_passages, b, a.total_passages, p0, p1);
  const int k = min(k1 - k0, a.k_max);
  const int P = min(min(p1 - p0, a.P_max), 64);
  // nothing of this question is read, or the block is past its rows
  if (k <= 0 || P <= 0 || rb * kEdRows >= k) return;
  const int c0 = s * kEdCols, ncol = min(kEdCols, a.d - c0);
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
  const int lane = tid & 63, l16 = lane & 15, kk = lane >> 4;
  const size_t zs = (size_t)b * a.S + s;
  const int tile0 = rb * kEdRows + 16 * w;         // first row of the wave's tile

  // The lane's row (rows past the question repeat its last row) and its
  // chunk of each group; chunks past the slice are zero.
  const int ri = min(tile0 + l16, k - 1);
  const int rid = a.kept_idx ? a.kept_idx[k0 + ri] : k0 + ri;
  const T* rsrc = rows + (a.kept_idx ? ((size_t)b * a.N + clampi(rid, 0, a.N - 1)) * a.d
                                     : (size_t)rid * a.d) + c0;
  // Keys of passages pt0 .. pt0 + 15 over the slice.  Float64 keys go
  // straight into LDS (direct loads, half a key row of 128 values per wave
  // instruction; wave w takes half rows w, w + 4, ...); caller-given f32 keys
  // pass through registers and are widened.  Passages past P repeat the last
  // one and columns past the slice repeat its last pair: their products
  // meet zero row values or are not written, and the key norms skip them.
  // The first keys (cached, shared by the question's workgroups) are
  // requested before the rows, so that they arrive first: the products then
  // start while the rows stream in, group by group.
  constexpr int KPT = kEdPT * kEdCols / 256;   // f32 key values per thread
  static_assert(KPT == kEdPT && kEdCols == 256, "thread t stages column t of each key");
  static_assert((kEdKeyStride * 8) % 16 == 0, "key rows start on 16 bytes");
  const bool dma = a.pkeys == nullptr;
  const uint32_t ks_lds = lds_addr(ks);
  float kf[KPT];
  auto load_keys = [&](int pt0) {
    if (dma) {
#pragma unroll
      for (int q = 0; q < 2 * kEdPT / 4; ++q) {
        const int hr = 4 * q + w, n = hr >> 1, h = hr & 1;
        const int col = min(h * 128 + 2 * lane, ncol - 2);
        lds_dma16(a.kbar + (size_t)(p0 + min(pt0 + n, P - 1)) * a.d + c0 + col,
                  __builtin_amdgcn_readfirstlane(ks_lds +
                                                 (uint32_t)(n * kEdKeyStride * 8 + h * 1024)));
      }
    } else {
      const int cc = min(tid, ncol - 1);
#pragma unroll
      for (int u = 0; u < KPT; ++u)
        kf[u] = a.pkeys[(size_t)(p0 + min(pt0 + u, P - 1)) * a.d + c0 + cc];
    }
  };
  auto store_keys = [&]() {
    if (!dma) {
#pragma unroll
      for (int u = 0; u < KPT; ++u) ks[u * kEdKeyStride + tid] = (double)kf[u];
    }
  };
  // (the row address first: waiting for its index later would also wait
  // for the direct key loads, which the compiler does not count)
  asm volatile("" : : "v"(rsrc) : "memory");
  load_keys(0);
  // bf16: every chunk of the slice in registers; f32 (twice the chunks):
  // each group's chunk is loaded where it is used
  constexpr bool kStage = sizeof(T) == 2;
  u32x4 x[kStage ? NG : 1];
  if (!kStage) {
  } else if (ncol == kEdCols) {
    // a whole slice: one base address, constant offsets
    const T* rl = rsrc + kk * E;
#pragma unroll
    for (int g = 0; g < NG; ++g) x[g] = *reinterpret_cast<const u32x4*>(rl + g * 4 * E);
  } else {
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int col = g * 4 * E + kk * E;
      x[g] = *reinterpret_cast<const u32x4*>(rsrc + (col < ncol ? col : 0));
    }
  }
  // the row loads stay above this point: the direct key loads, issued
  // before them, are complete once at most their count is pending
  asm volatile("" ::: "memory");
  if (dma) wait_vmcnt<kStage ? NG : 0>();
  store_keys();

  double qq = 0.0;
  for (int pt0 = 0; pt0 < P; pt0 += kEdPT) {
    if (pt0 > 0) {
      __syncthreads();                             // the previous keys are read
      load_keys(pt0);
      if (dma) wait_vmcnt<0>();
      store_keys();
    }
    __syncthreads();
    if (rb == 0) {
      // |k̄_j|^2 over the slice: wave w takes passages w, w + 4, w + 8,
      // w + 12, lane l the columns l, l + 64, ... in order, then a fixed
      // shuffle tree
      double q2[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const double* kr = ks + (w + 4 * u) * kEdKeyStride;
        q2[u] = 0.0;
#pragma unroll
        for (int c = lane; c < kEdCols; c += 64)
          if (c < ncol) q2[u] = fma(kr[c], kr[c], q2[u]);
      }
#pragma unroll
      for (int sh = 32; sh >= 1; sh >>= 1)
#pragma unroll
        for (int u = 0; u < 4; ++u) q2[u] += __shfl_xor(q2[u], sh, kWave);
      if (lane == 0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int j = pt0 + w + 4 * u;
          if (j < P) a.kn2p[zs * a.P_max + j] = q2[u];
        }
      }
    }
    // products: per group, E key values and the lane's chunk; four
    // independent accumulators (MFMA m goes to m % 4), added in order
    f64x4_t acc[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = f64x4_t{0.0, 0.0, 0.0, 0.0};
    const double* kp = ks + l16 * kEdKeyStride + kk * E;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      double kv[E], qa[E];
#pragma unroll
      for (int m = 0; m < E; m += 2) {
        const double2 k2 = *reinterpret_cast<const double2*>(kp + g * 4 * E + m);
        kv[m] = k2.x;
        kv[m + 1] = k2.y;
      }
      // a chunk past the slice holds 0 (its load read the first chunk); the
      // conversion stays inside the passage loop (an empty asm redefines the
      // chunk), so only one group's values are live at a time
      const int col = g * 4 * E + kk * E;
      u32x4 xg;
      if constexpr (kStage) {
        xg = x[g];
      } else {
        // (the base passes through an empty asm so that the compiler forms
        // each address here instead of keeping all of them live)
        const T* rp = rsrc;
        int lim = ncol;
        asm volatile("" : "+v"(rp), "+v"(lim));
        xg = *reinterpret_cast<const u32x4*>(rp + (col < lim ? col : 0));
      }
      if (col >= ncol) xg = u32x4{0u, 0u, 0u, 0u};
      asm volatile("" : "+v"(xg));
      unpack16_f64<T>(xg, qa);
#pragma unroll
      for (int m = 0; m < E; ++m)
        acc[m & 3] = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[m], kv[m], acc[m & 3], 0, 0, 0);
      if (pt0 == 0) {
#pragma unroll
        for (int m = 0; m < E; ++m) qq = fma(qa[m], qa[m], qq);
      }
      // one group's key reads and conversions in flight at a time (keeps
      // the register count at three waves per SIMD)
      __builtin_amdgcn_sched_barrier(0);
    }
    // D[i][j]: register v of lane l holds row 4v + l/16 of the tile, passage l % 16
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = tile0 + 4 * v + kk, j = pt0 + l16;
      if (i < k && j < P)
        a.part[(zs * a.k_max + i) * a.P_max + j] = ((acc[0][v] + acc[1][v]) + acc[2][v]) + acc[3][v];
    }
  }
  // lanes l16, l16 + 16, l16 + 32, l16 + 48 hold the four column slots of row l16
  qq += __shfl_xor(qq, 16, kWave);
  qq += __shfl_xor(qq, 32, kWave);
  if (kk == 0 && tile0 + l16 < k) a.qn2p[zs * a.k_max + tile0 + l16] = qq;
}

// ---------------------------------------------------------------------------
// Edge selection, one workgroup per question.
constexpr int kGSelThreads = 1024;

// The attention's work list, built by one extra workgroup of the selection
// launch (items NULL: none).
struct PlanArgs {
  int4* items;
  const int32_t* passage_offsets;
  int H, total_tokens, n_ids;
};
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

// Candidate keys, one thread per (row, passage) of a question: the slice
// partials of the dot product (and of both squared norms) summed in slice
// order, the cosine (or the scaled dot product) formed from them, and its
// order-preserving key written over slice 0 of the partials; a passage the
// verification gate dropped gets the lowest key.  Each candidate's partials
// are read and its key written by one thread only.
__global__ void __launch_bounds__(256)
edge_keys_kernel(double* __restrict__ part, const double* __restrict__ qn2p,
                 const double* __restrict__ kn2p, int S,
                 const int32_t* __restrict__ kept_offsets,
                 const int32_t* __restrict__ query_passages, int total_kept,
                 int total_passages, int k_max, int P_max, int d, int metric,
                 const uint8_t* __restrict__ keep) {
  const int b = blockIdx.y;
  int k0, k1, p0, p1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  range_of(query_passages, b, total_passages, p0, p1);
  const int k = min(k1 - k0, k_max);
  const int P = min(min(p1 - p0, P_max), 64);
  const int n = min(k * P, kGSelThreads * kGSelMaxPT);
  const int f = blockIdx.x * blockDim.x + threadIdx.x;
  if (f >= n) return;
  const int i = f / P, j = f - i * P;
  // sum of S values at base + s * stride, in slice order (slices clamped
  // into range, so that every load of a batch is unconditional)
  auto slice_sum = [&](const double* base, size_t stride) -> double {
    double acc = 0.0;
    for (int sl0 = 0; sl0 < S; sl0 += 16) {
      double x[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) x[u] = base[(size_t)min(sl0 + u, S - 1) * stride];
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (sl0 + u < S) acc += x[u];
    }
    return acc;
  };
  double* cand = part + ((size_t)b * S * k_max + i) * P_max + j;
  const double dot = slice_sum(cand, (size_t)k_max * P_max);
  double c;
  if (metric == SKIP_EDGE_DOT) {
    c = dot * (1.0 / sqrt((double)d));
  } else {
    const double nq = sqrt(slice_sum(qn2p + (size_t)b * S * k_max + i, (size_t)k_max));
    const double nk = sqrt(slice_sum(kn2p + (size_t)b * S * P_max + j, (size_t)P_max));
    c = (nq > 0.0 && nk > 0.0) ? dot / (nq * nk) : 0.0;
  }
  const bool kept = keep ? keep[p0 + j] != 0 : true;
  *reinterpret_cast<uint64_t*>(cand) = kept ? order_key(c) : 0ull;
}

__global__ void __launch_bounds__(kGSelThreads)
edge_select_kernel(const double* __restrict__ part, int S,
                   const int32_t* __restrict__ kept_offsets,
                   const int32_t* __restrict__ query_passages, int B, int total_kept,
                   int total_passages, int k_max, int P_max, double avg_degree,
                   int rule, double beta, const uint8_t* __restrict__ keep,
                   uint64_t* __restrict__ rowmask, int32_t* __restrict__ rowptr_out,
                   int32_t* __restrict__ col_out, PlanArgs plan) {
  __shared__ SelectShared sh;
  __shared__ uint32_t scan_sh[20];
  __shared__ uint8_t flag[kGSelThreads * kGSelMaxPT];
  // the keys of the per-row cut (the work list builder's LDS in the extra
  // workgroup)
  __shared__ __align__(16) uint64_t rkeys[kGSelThreads * kGSelMaxPT];
  static_assert(sizeof(PlanLds) <= sizeof(rkeys), "the work list builder reuses the key LDS");
  if ((int)blockIdx.x == B) {
    // the extra workgroup: the attention's work list (it depends on the
    // offsets only)
    build_attention_plan(*reinterpret_cast<PlanLds*>(rkeys), scan_sh, kept_offsets,
                         query_passages, plan.passage_offsets, B, plan.H, total_kept,
                         total_passages, plan.total_tokens, k_max, P_max, plan.n_ids,
                         plan.items);
    return;
  }
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

  const int C = (n + blockDim.x - 1) / blockDim.x;
  const int e0 = threadIdx.x * C;
  const int cnt = max(0, min(C, n - e0));
  // the candidates' keys, formed by the key launch over slice 0 of the
  // partials
  const uint64_t* ck = reinterpret_cast<const uint64_t*>(part) + (size_t)b * S * k_max * P_max;
  uint64_t keys[kGSelMaxPT];
#pragma unroll
  for (int jj = 0; jj < kGSelMaxPT; ++jj) {
    keys[jj] = 0ull;
    if (jj < cnt) {
      const int f = e0 + jj, ii = f / P;
      keys[jj] = ck[(size_t)ii * P_max + (f - ii * P)];
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
    flags = block_select_top_wide<kGSelMaxPT>(keys, cnt, n, E, &sh);
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

int edge_slices(const skip_problem_t& p) { return (p.d + kEdCols - 1) / kEdCols; }

hipError_t launch_edge_dot(const skip_problem_t& p, QuerySource q,
                           const int32_t* kept_offsets, const int32_t* query_passages,
                           const double* kbar, const float* passage_keys, EdgePartials ep,
                           hipStream_t s) {
  if (p.k_max <= 0 || p.P_max <= 0) return hipSuccess;
  EdgeDotArgs a;
  a.kept_idx = q.kept_idx;
  a.N = q.N;
  a.kept_offsets = kept_offsets;
  a.query_passages = query_passages;
  a.kbar = kbar;
  a.pkeys = passage_keys;
  a.d = p.d;
  a.total_kept = p.total_kept;
  a.total_passages = p.total_passages;
  a.k_max = p.k_max;
  a.P_max = p.P_max;
  a.B = p.B;
  a.S = edge_slices(p);
  a.RB = (p.k_max + kEdRows - 1) / kEdRows;
  a.part = ep.part;
  a.qn2p = ep.qn2;
  a.kn2p = ep.kn2;
  const long long nwg = 8ll * ((p.B + 7) / 8) * a.S * a.RB;
  if (nwg > INT32_MAX) return hipErrorInvalidValue;
  dim3 grid((unsigned)nwg);
  if (p.dtype == SKIP_F32)
    hipLaunchKernelGGL(edge_dot_kernel<float>, grid, dim3(256), 0, s, (const float*)q.base, a);
  else
    hipLaunchKernelGGL(edge_dot_kernel<bf16_t>, grid, dim3(256), 0, s, (const bf16_t*)q.base, a);
  return hipGetLastError();
}

hipError_t launch_edge_select(const skip_problem_t& p, EdgePartials ep,
                              const int32_t* kept_offsets, const int32_t* query_passages,
                              uint64_t* rowmask, int32_t* rowptr_out, int32_t* col_out,
                              hipStream_t s, const uint8_t* passage_keep,
                              const int32_t* passage_offsets, int32_t* plan) {
  PlanArgs pa{};
  const long long n_ids = plan ? attn_plan_ids(p) : 0;
  if (n_ids > INT32_MAX / 16) return hipErrorInvalidValue;
  if (n_ids > 0) {
    pa.items = reinterpret_cast<int4*>(plan);
    pa.passage_offsets = passage_offsets;
    pa.H = p.H;
    pa.total_tokens = p.total_tokens;
    pa.n_ids = (int)n_ids;
  }
  const int S = edge_slices(p);
  if (p.total_kept > 0 && p.k_max > 0 && p.P_max > 0) {
    // the candidates' keys from the partials of the dot-product launch
    const int n = (int)std::min<long long>((long long)p.k_max * std::min(p.P_max, 64),
                                           (long long)kGSelThreads * kGSelMaxPT);
    hipLaunchKernelGGL(edge_keys_kernel, dim3((n + 255) / 256, p.B), dim3(256), 0, s, ep.part,
                       ep.qn2, ep.kn2, S, kept_offsets, query_passages, p.total_kept,
                       p.total_passages, p.k_max, p.P_max, p.d, p.edge_metric, passage_keep);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(edge_select_kernel, dim3(p.B + (n_ids > 0 ? 1 : 0)), dim3(kGSelThreads),
                     0, s, ep.part, S, kept_offsets, query_passages, p.B, p.total_kept,
                     p.total_passages, p.k_max, p.P_max, p.avg_degree, p.edge_rule,
                     p.edge_beta, passage_keep, rowmask, rowptr_out, col_out, pa);
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

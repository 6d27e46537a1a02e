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
#include "skip_plan.h"
#include "skip_pool.h"
#include "skip_select.h"

namespace skip {

// ---------------------------------------------------------------------------
// Edge dot products on the float64 matrix cores, split over d.
// Workgroup = (256-column slice, question), one workgroup per CU over the
// chip for the usual shapes; the slices of a question run on one XCD
// (workgroup id L goes to XCD L % 8).  v_mfma_f64_16x16x4_f64 takes one
// element of A (16 rows x 4 columns) and one of B (4 columns x 16 passages)
// per lane: lane l supplies row/passage l % 16 and column slot l / 16.  The
// contraction order over columns is free, so column slot kk of MFMA m within
// a group of 4·E columns (E = 8 bf16 or 4 f32 per 16-byte chunk) is column
// E*kk + m: a lane then reads one 16-byte chunk of its row and E consecutive
// key values per group.
//   * The kept rows come into LDS in blocks of 192 (16-row tiles; wave w
//     takes tiles w, w + 4, w + 8) by direct loads of whole 512-byte row
//     slices (f32 rows in two 128-column passes); chunk c of row r sits at
//     slot c ^ (r & 7), so that the lanes' reads of one chunk group fall on
//     distinct banks.  Chunks past the slice are cleared.
//   * The passage keys of the slice sit in LDS as float64, 16 passages at a
//     time, read by all four waves.
// Each lane also sums the squares of its row values (partial row norms); the
// key norms come from the keys in LDS.  Results per slice are summed in slice
// order by the selection kernel.
constexpr int kEdCols = 256;               // columns per slice
constexpr int kEdBlockRows = 192;          // rows per LDS block (12 tiles)
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
  int d, total_kept, total_passages, k_max, P_max, B, S;
  double* part;                // [B][S][k_max][P_max] partial <q_i, k̄_j>
  double* qn2p;                // [B][S][k_max]        partial |q_i|^2
  double* kn2p;                // [B][S][P_max]        partial |k̄_j|^2
};

template <typename T>
__global__ void __launch_bounds__(256)
edge_dot_kernel(const T* __restrict__ rows, EdgeDotArgs a) {
  constexpr int E = 16 / (int)sizeof(T);          // columns per 16-byte chunk
  constexpr int CPP = 32 * E;                      // columns per pass (512 bytes of a row)
  constexpr int NP = kEdCols / CPP;                // passes per slice
  __shared__ __align__(16) uint8_t rbuf[kEdBlockRows * 512];
  __shared__ __align__(16) double ks[kEdPT * kEdKeyStride];
  const int L = blockIdx.x, xcd = L & 7, jl = L >> 3;
  const int s = jl % a.S, b = xcd + 8 * (jl / a.S), tid = threadIdx.x;
  if (b >= a.B) return;
  int k0, k1, p0, p1;
  range_of(a.kept_offsets, b, a.total_kept, k0, k1);
  range_of(a.query_passages, b, a.total_passages, p0, p1);
  const int k = min(k1 - k0, a.k_max);
  const int P = min(min(p1 - p0, a.P_max), 64);
  if (k <= 0 || P <= 0) return;                  // nothing of this question is read
  const int c0 = s * kEdCols, ncol = min(kEdCols, a.d - c0);
  const int w = tid >> 6, lane = tid & 63, l16 = lane & 15, kk = lane >> 4;
  const uint32_t rlds = lds_addr(rbuf);
  const size_t zs = (size_t)b * a.S + s;

  // Copy rows blk0 .. blk0 + 191, columns [pass·CPP, pass·CPP + CPP) of the
  // slice, into rbuf.  Wave w copies rows 48w .. 48w + 47, two per load
  // instruction: lane l writes slot l % 32 of row 2j + l / 32, which holds
  // chunk (l % 32) ^ (row & 7).  Rows past the question repeat its last row;
  // chunks past the slice read its first chunk (cleared afterwards).  The
  // row indices are all read before the first copy: the copies are opaque to
  // the compiler, which would otherwise wait for each one before the next.
  auto stage_rows = [&](int blk0, int pass) {
    const int half = lane >> 5, slot = lane & 31;
    int rid[24];
#pragma unroll
    for (int j = 0; j < 24; ++j) {
      const int i = min(blk0 + 48 * w + 2 * j + half, k - 1);
      rid[j] = a.kept_idx ? a.kept_idx[k0 + i] : k0 + i;
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < 24; ++j) {
      const int r = 48 * w + 2 * j + half;         // row within the block
      const int col = pass * CPP + (slot ^ (r & 7)) * E;
      const int colc = col < ncol ? col : 0;
      const size_t row = a.kept_idx ? (size_t)b * a.N + clampi(rid[j], 0, a.N - 1)
                                    : (size_t)rid[j];
      lds_dma16(rows + row * a.d + c0 + colc,
               __builtin_amdgcn_readfirstlane(rlds + (uint32_t)(48 * w + 2 * j) * 512u));
    }
  };
  // after the copies of a pass have landed: clear the chunks past the slice
  // (each wave its own rows; every wave waits for its copies first)
  auto finish_rows = [&](int pass) {
    wait_vmcnt<0>();
    if (pass * CPP + CPP > ncol) {
      for (int t = lane; t < 48 * 32; t += 64) {
        const int r = 48 * w + (t >> 5), sl = t & 31;
        if (pass * CPP + (sl ^ (r & 7)) * E >= ncol)
          *reinterpret_cast<u32x4*>(rbuf + r * 512 + sl * 16) = u32x4{0u, 0u, 0u, 0u};
      }
    }
    __syncthreads();                               // rows of every wave are in
  };

  for (int blk0 = 0; blk0 < k; blk0 += kEdBlockRows) {
    for (int pt0 = 0; pt0 < P; pt0 += kEdPT) {
      // two accumulators per tile (even and odd MFMA of a group), added at
      // the end: six independent chains keep the matrix pipeline busy
      double qq[3] = {0.0, 0.0, 0.0};
      f64x4_t acc[3][2];
#pragma unroll
      for (int t = 0; t < 3; ++t) acc[t][0] = acc[t][1] = f64x4_t{0.0, 0.0, 0.0, 0.0};
      for (int pass = 0; pass < NP; ++pass) {
        __syncthreads();                           // the previous rows and keys are read
        stage_rows(blk0, pass);
        // keys of passages pt0 .. pt0 + 15 over this pass's columns (0 past P
        // or the slice), under the row copies
        // (every load unconditional, passages and columns clamped into range
        // and the value replaced by 0 afterwards, so that they all issue
        // before the first wait)
        {
          constexpr int KPT = kEdPT * CPP / 256;   // key values per thread
          double kvv[KPT];
#pragma unroll
          for (int u = 0; u < KPT; ++u) {
            const int t = tid + 256 * u, n = t / CPP, c = pass * CPP + t % CPP;
            const size_t o = (size_t)(p0 + min(pt0 + n, P - 1)) * a.d + c0 + min(c, ncol - 1);
            kvv[u] = a.pkeys ? (double)a.pkeys[o] : a.kbar[o];
          }
#pragma unroll
          for (int u = 0; u < KPT; ++u) {
            const int t = tid + 256 * u, n = t / CPP, c = pass * CPP + t % CPP;
            ks[n * kEdKeyStride + c] = (pt0 + n < P && c < ncol) ? kvv[u] : 0.0;
          }
        }
        finish_rows(pass);
        if (blk0 == 0) {
          // |k̄_j|^2 over the pass's columns: wave w takes passages w, w + 4,
          // w + 8, w + 12, lane l the columns l, l + 64, ... in order, then a
          // fixed shuffle tree; added to the partial of the previous pass
          double q2[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const double* kr = ks + (w + 4 * u) * kEdKeyStride + pass * CPP;
            q2[u] = 0.0;
            for (int c = lane; c < CPP; c += 64) q2[u] = fma(kr[c], kr[c], q2[u]);
          }
#pragma unroll
          for (int sh = 32; sh >= 1; sh >>= 1)
#pragma unroll
            for (int u = 0; u < 4; ++u) q2[u] += __shfl_xor(q2[u], sh, kWave);
          if (lane == 0) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              const int j = pt0 + w + 4 * u;
              if (j < P) {
                double* o = a.kn2p + zs * a.P_max + j;
                *o = (pass == 0 ? 0.0 : *o) + q2[u];
              }
            }
          }
        }
        // products: per group of 4 chunks, one key read (E values) feeds the
        // three row tiles of the wave
        const double* kp = ks + l16 * kEdKeyStride + pass * CPP + kk * E;
#pragma unroll 2
        for (int g = 0; g < 8; ++g) {
          double kv[E];
#pragma unroll
          for (int m = 0; m < E; ++m) kv[m] = kp[g * 4 * E + m];
          double qa[3][8];
#pragma unroll
          for (int t = 0; t < 3; ++t) {
            const int r = 16 * (w + 4 * t) + l16;          // row within the block
            const u32x4 x = *reinterpret_cast<const u32x4*>(
                rbuf + r * 512 + (((4 * g + kk) ^ (r & 7)) * 16));
            unpack16_f64<T>(x, qa[t]);
          }
#pragma unroll
          for (int m = 0; m < E; ++m)
#pragma unroll
            for (int t = 0; t < 3; ++t)
              acc[t][m & 1] = __builtin_amdgcn_mfma_f64_16x16x4f64(qa[t][m], kv[m], acc[t][m & 1], 0, 0, 0);
          if (pt0 == 0) {
#pragma unroll
            for (int t = 0; t < 3; ++t)
#pragma unroll
              for (int m = 0; m < E; ++m) qq[t] = fma(qa[t][m], qa[t][m], qq[t]);
          }
        }
      }
      // D[i][j]: register v of lane l holds row 4v + l/16 of the tile, passage l % 16
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const int tile0 = blk0 + 16 * (w + 4 * t);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int i = tile0 + 4 * v + kk, j = pt0 + l16;
          if (i < k && j < P) a.part[(zs * a.k_max + i) * a.P_max + j] = acc[t][0][v] + acc[t][1][v];
        }
        if (pt0 == 0) {
          // lanes l16, l16 + 16, l16 + 32, l16 + 48 hold the four column slots of row l16
          double q = qq[t];
          q += __shfl_xor(q, 16, kWave);
          q += __shfl_xor(q, 32, kWave);
          const int i = tile0 + l16;
          if (kk == 0 && i < k) a.qn2p[zs * a.k_max + i] = q;
        }
      }
    }
  }
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

__global__ void __launch_bounds__(kGSelThreads)
edge_select_kernel(const double* __restrict__ part, const double* __restrict__ qn2p,
                   const double* __restrict__ kn2p, int S,
                   const int32_t* __restrict__ kept_offsets,
                   const int32_t* __restrict__ query_passages, int B, int total_kept,
                   int total_passages, int k_max, int P_max, int d, double avg_degree,
                   int rule, int metric, double beta, const uint8_t* __restrict__ keep,
                   uint64_t* __restrict__ rowmask, int32_t* __restrict__ rowptr_out,
                   int32_t* __restrict__ col_out, PlanArgs plan) {
  __shared__ SelectShared sh;
  __shared__ uint32_t scan_sh[20];
  __shared__ uint8_t flag[kGSelThreads * kGSelMaxPT];
  // row norms while the keys are formed, then the keys of the per-row cut
  __shared__ __align__(16) uint64_t rkeys[kGSelThreads * kGSelMaxPT];
  __shared__ double knorm[64];
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
  double* qnorm = reinterpret_cast<double*>(rkeys);
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
  // Norms |q_i| and |k̄_j| first: square roots of the slice partials summed
  // in slice order (slices clamped into range, so every load of a batch is
  // unconditional), kept in LDS.
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
  if (metric != SKIP_EDGE_DOT) {
    const int kr = min(k, kGSelThreads * kGSelMaxPT);   // rows that have candidates
    for (int t = threadIdx.x; t < kr + P; t += blockDim.x) {
      if (t < kr) qnorm[t] = sqrt(slice_sum(qn2p + (size_t)b * S * k_max + t, (size_t)k_max));
      else knorm[t - kr] = sqrt(slice_sum(kn2p + (size_t)b * S * P_max + (t - kr), (size_t)P_max));
    }
    __syncthreads();
  }
  // compatibility of (i, j) from the per-slice partial products, in slice
  // order; two candidates at a time, sixteen slices of their loads in flight
  uint64_t keys[kGSelMaxPT];
#pragma unroll
  for (int jj = 0; jj < kGSelMaxPT; ++jj) keys[jj] = 0ull;
#pragma unroll
  for (int jj = 0; jj < kGSelMaxPT; jj += 2) {
    if (jj < cnt) {
      int ii[2], pj[2];
      double dot[2] = {0.0, 0.0};
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int f = min(e0 + jj + h, n - 1);
        ii[h] = f / P;
        pj[h] = f - ii[h] * P;
      }
      for (int sl0 = 0; sl0 < S; sl0 += 16) {
        double pd[2][16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const size_t base = (size_t)b * S + min(sl0 + u, S - 1);
#pragma unroll
          for (int h = 0; h < 2; ++h) pd[h][u] = part[(base * k_max + ii[h]) * P_max + pj[h]];
        }
#pragma unroll
        for (int u = 0; u < 16; ++u)
          if (sl0 + u < S) {
#pragma unroll
            for (int h = 0; h < 2; ++h) dot[h] += pd[h][u];
          }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        if (jj + h < cnt) {
          double c;
          if (metric == SKIP_EDGE_DOT) {
            c = dot[h] * inv_sqrt_d;
          } else {
            const double nq = qnorm[ii[h]], nk = knorm[pj[h]];
            c = (nq > 0.0 && nk > 0.0) ? dot[h] / (nq * nk) : 0.0;
          }
          keys[jj + h] = ((pkeep >> pj[h]) & 1ull) ? order_key(c) : 0ull;
        }
      }
    }
  }
  __syncthreads();                 // the row norms are read before rkeys is written
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
  a.part = ep.part;
  a.qn2p = ep.qn2;
  a.kn2p = ep.kn2;
  dim3 grid(8 * ((p.B + 7) / 8) * a.S);
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
  hipLaunchKernelGGL(edge_select_kernel, dim3(p.B + (n_ids > 0 ? 1 : 0)), dim3(kGSelThreads),
                     0, s, ep.part, ep.qn2, ep.kn2, edge_slices(p), kept_offsets,
                     query_passages, p.B, p.total_kept, p.total_passages, p.k_max, p.P_max, p.d,
                     p.avg_degree, p.edge_rule, p.edge_metric, p.edge_beta, passage_keep,
                     rowmask, rowptr_out, col_out, pa);
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

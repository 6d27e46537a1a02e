// Regions of the kept tokens (paper Sec. 3.4: region-conditional retrieval
// clusters the kept visual tokens into R = min(V'/4, 8) regions by an
// approximate k-means in embedding space; each region's centroid then seeds a
// retrieval query).  Lloyd iterations from a fixed start, float64 throughout:
//   start       centroid r = kept row floor((2r+1) k / (2R))
//   iteration   each row to the nearest centroid (squared distance, ties to
//               the lower region); each centroid to the mean of its rows, a
//               region without rows keeping its centroid
// Launches: one clear of the per-question counters, then n_iter + 1 steps of
// region_step_kernel over (column slice, question) workgroups:
//   step 0          start centroids; partial products for the first assignment
//   step t (< n)    centroids from assignment t; partial products for t + 1
//   step n          centroids from assignment n; outputs
// In a step the slice workgroups of a question write their partial dot
// products v_i . c_r and squared norms |c_r|^2 over their columns (coherent
// stores); the last of them to finish (a counter) sums the partials in slice
// order and assigns
// every row by argmin_r |c_r|^2 - 2 v_i . c_r, which is |v_i - c_r|^2 less the
// row's own |v_i|^2.
#include "skip_common.h"
#include "skip_internal.h"

namespace skip {

constexpr int kRegCols = 256;     // columns per slice = threads per workgroup
constexpr int kRegMax = 16;       // largest r_max
constexpr int kRegMaxRows = 16384; // largest k_max

namespace {

template <typename T> __device__ __forceinline__ double reg_load1(const T* p);
template <> __device__ __forceinline__ double reg_load1<float>(const float* p) {
  return (double)*p;
}
template <> __device__ __forceinline__ double reg_load1<bf16_t>(const bf16_t* p) {
  return (double)bf16_to_f32(*p);
}

// eight consecutive elements as doubles (16-byte aligned for bf16, 32 for f32)
template <typename T> __device__ __forceinline__ void reg_load8(const T* p, double* o);
template <> __device__ __forceinline__ void reg_load8<float>(const float* p, double* o) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}
template <> __device__ __forceinline__ void reg_load8<bf16_t>(const bf16_t* p, double* o) {
  const u32x4 x = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    o[2 * w] = (double)__uint_as_float(x[w] << 16);
    o[2 * w + 1] = (double)__uint_as_float(x[w] & 0xffff0000u);
  }
}

__device__ __forceinline__ int regions_of(int k, int r_max) {
  if (k <= 0) return 0;
  const int r = k / 4;
  return r < 1 ? 1 : (r > r_max ? r_max : r);
}

}  // namespace

__global__ void region_clear_kernel(int32_t* __restrict__ done, int B) {
  for (int b = threadIdx.x; b < B; b += blockDim.x) done[b] = 0;
}

struct RegionArgs {
  const int32_t* kept_offsets;
  const int32_t* kept_idx;     // NULL: rows are the kept rows themselves
  int N, total_kept, B, d, k_max, r_max, S, t, n_iter;
  double* C;                   // [B][r_max][d]      centroids of the last step
  double* P;                   // [B][S][k_max][r_max] partial v_i . c_r
  double* CN;                  // [B][S][r_max]       partial |c_r|^2
  uint8_t* asg;                // [total_kept]        current assignment
  int32_t* perm;               // [total_kept]        row ids sorted by region (stable)
  uint8_t* sreg;               // [total_kept]        region of each sorted position
  int32_t* sizes;              // [B][r_max]          rows per region
  int32_t* done;               // [B]                 finished slices
  int32_t* region_out;         // [total_kept]
  float* cent_out;             // [B][r_max][d]
  int32_t* sizes_out;          // [B][r_max] or NULL
};

// 8 consecutive elements of a row (16-byte aligned for bf16, 32 for f32) as
// raw words, converted when used
template <typename T> struct RegChunk;
template <> struct RegChunk<bf16_t> {
  u32x4 w;
  __device__ __forceinline__ void load(const bf16_t* p) { w = *reinterpret_cast<const u32x4*>(p); }
  __device__ __forceinline__ double at(int e) const {
    const uint32_t x = w[e >> 1];
    return (double)__uint_as_float((e & 1) ? (x & 0xffff0000u) : (x << 16));
  }
};
template <> struct RegChunk<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = *reinterpret_cast<const float4*>(p);
    b = *reinterpret_cast<const float4*>(p + 4);
  }
  __device__ __forceinline__ double at(int e) const {
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    return (double)v[e];
  }
};

constexpr int kRegRowBatch = 32;   // rows whose loads are issued together (update)
// columns of a row slice loaded at once (dots): the whole bf16 slice, half of
// an f32 one
template <typename T> struct RegLoadCols { static constexpr int n = 128; };
template <> struct RegLoadCols<bf16_t> { static constexpr int n = 256; };
constexpr int kRegPairs = 4;       // (row, region) sums per thread at once (assignment)

// RM: a compile-time bound on the regions (4, 8 or 16), so that every loop
// over the regions unrolls and the per-region sums stay in fixed registers
// (a run-time bound made the compiler index the register file, one
// instruction at a time).
template <typename T, bool IDX, int RM>
__global__ void __launch_bounds__(kRegCols)
region_step_kernel(const T* __restrict__ rows, RegionArgs a) {
  __shared__ double cs[kRegMax][kRegCols];      // this step's centroids, this slice
  __shared__ __align__(16) double dl[kRegCols * kRegMax];     // distances of a block of rows (last slice)
  __shared__ int last;
  __shared__ int cnt[kRegMax];
  __shared__ __align__(16) uint8_t asl[kRegMaxRows];          // assignment (last slice) / sorted regions (update)
  // All slices of a question run on one XCD (workgroup id L goes to XCD
  // L % 8): its L2 then holds the question's whole kept rows across the
  // steps.  With slices spread over the XCDs instead, every XCD would hold
  // the same few column slices of all questions, and rows 8 KiB apart map
  // those slices onto a small fraction of the L2 sets.
  const int L = blockIdx.x, xcd = L & 7, jl = L >> 3;
  const int s = jl % a.S, b = xcd + 8 * (jl / a.S), tid = threadIdx.x;
  if (b >= a.B) return;
  int k0, k1;
  range_of(a.kept_offsets, b, a.total_kept, k0, k1);
  const int k = min(k1 - k0, a.k_max);
  const int R = regions_of(k, a.r_max);
  const int c0 = s * kRegCols, c = c0 + tid;
  const int ncol = min(kRegCols, a.d - c0);
  const bool cok = tid < ncol;
  // row i of the question: V[b][kept_idx[k0+i]] (IDX) or rows[k0+i]
  auto row_id = [&](int i) -> size_t {
    if (IDX) return (size_t)b * a.N + clampi(a.kept_idx[k0 + i], 0, a.N - 1);
    return (size_t)(k0 + i);
  };
  auto row_of = [&](int i) -> const T* { return rows + row_id(i) * a.d; };
  const bool final_step = a.t == a.n_iter;

  if (R == 0) {
    if (final_step) {
      for (int r = 0; r < a.r_max; ++r)
        if (cok) a.cent_out[((size_t)b * a.r_max + r) * a.d + c] = 0.f;
      if (s == 0 && a.sizes_out && tid < a.r_max) a.sizes_out[b * a.r_max + tid] = 0;
    }
    return;
  }

  // ---- centroids of this step, this slice's columns (thread = column)
  if (a.t == 0) {
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      if (r < R) {
        const int pos = ((2 * r + 1) * k) / (2 * R);
        cs[r][tid] = cok ? reg_load1<T>(row_of(pos) + c) : 0.0;
      }
    }
  } else {
    // the rows sorted by region (perm: row ids, ascending within a region;
    // sreg: the region of each sorted position) are summed in one pass:
    // each thread keeps its column's running sum in a register and hands it
    // to LDS where the region changes (a uniform test).  Row ids and regions
    // are staged in LDS 8192 at a time; 32 row loads are issued together
    // (positions and columns clamped into range, so every load is
    // unconditional).  Regions without rows keep their centroid.
    for (int r = tid; r < R; r += blockDim.x) cnt[r] = a.sizes[b * a.r_max + r];
    int* ids = reinterpret_cast<int*>(dl);
    constexpr int kIds = (int)(sizeof(dl) / (sizeof(int)));
    const int cc = cok ? c : c0;
    int cur = -1;
    double acc = 0.0;
    for (int g0 = 0; g0 < k; g0 += kIds) {
      const int ng = min(kIds, k - g0);
      const int ng32 = (ng + kRegRowBatch - 1) / kRegRowBatch * kRegRowBatch;
      __syncthreads();                 // the previous group is consumed
      // Padding up to a whole batch repeats the last row id (an in-range
      // load) and marks its region 0xff (skipped).
      for (int j = tid; j < ng32; j += blockDim.x) {
        const int jj = min(j, ng - 1);
        ids[j] = a.perm[k0 + g0 + jj];
        asl[j] = (j < ng) ? a.sreg[k0 + g0 + jj] : (uint8_t)0xff;
      }
      __syncthreads();
      for (int j0 = 0; j0 < ng; j0 += kRegRowBatch) {
        double v[kRegRowBatch];
        int4 id4[kRegRowBatch / 4];
        uint32_t rg4[kRegRowBatch / 4];
#pragma unroll
        for (int q = 0; q < kRegRowBatch / 4; ++q) {
          id4[q] = *reinterpret_cast<const int4*>(&ids[j0 + 4 * q]);
          rg4[q] = *reinterpret_cast<const uint32_t*>(&asl[j0 + 4 * q]);
        }
#pragma unroll
        for (int q = 0; q < kRegRowBatch / 4; ++q) {
          v[4 * q + 0] = reg_load1<T>(rows + (size_t)id4[q].x * a.d + cc);
          v[4 * q + 1] = reg_load1<T>(rows + (size_t)id4[q].y * a.d + cc);
          v[4 * q + 2] = reg_load1<T>(rows + (size_t)id4[q].z * a.d + cc);
          v[4 * q + 3] = reg_load1<T>(rows + (size_t)id4[q].w * a.d + cc);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int u = 0; u < kRegRowBatch; ++u) {
          const int rg = (int)((rg4[u / 4] >> (8 * (u % 4))) & 0xffu);
          if (rg != 0xff) {
            if (rg != cur) {
              if (cur >= 0) cs[cur][tid] = acc;
              acc = 0.0;
              cur = rg;
            }
            acc += v[u];
          }
        }
      }
    }
    if (cur >= 0) cs[cur][tid] = acc;
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      if (r < R) {
        const int n = cnt[r];
        if (n > 0) cs[r][tid] = cok ? cs[r][tid] / (double)n : 0.0;
        else cs[r][tid] = cok ? a.C[((size_t)b * a.r_max + r) * a.d + c] : 0.0;
      }
    }
    __syncthreads();        // cnt and the LDS staging buffers are reused below
  }
  if (!final_step && cok) {
    for (int r = 0; r < R; ++r) a.C[((size_t)b * a.r_max + r) * a.d + c] = cs[r][tid];
  }
  __syncthreads();

  if (final_step) {
    for (int r = 0; r < a.r_max; ++r)
      if (cok)
        a.cent_out[((size_t)b * a.r_max + r) * a.d + c] = r < R ? (float)cs[r][tid] : 0.f;
    if (s == 0) {
      for (int i = tid; i < k; i += blockDim.x) a.region_out[k0 + i] = a.asg[k0 + i];
      if (a.sizes_out && tid < a.r_max)
        a.sizes_out[b * a.r_max + tid] = tid < R ? a.sizes[b * a.r_max + tid] : 0;
    }
    return;
  }

  // ---- partial products over this slice: thread = row; each 128-column half
  // of the row's slice is loaded whole before its products
  double* P = a.P + ((size_t)b * a.S + s) * a.k_max * a.r_max;
  for (int i = tid; i < k; i += blockDim.x) {
    const T* v = row_of(i) + c0;
    double dot[RM];
#pragma unroll
    for (int r = 0; r < RM; ++r) dot[r] = 0.0;
    constexpr int kHalf = RegLoadCols<T>::n;
    for (int h0 = 0; h0 < ncol; h0 += kHalf) {
      RegChunk<T> ch[kHalf / 8];
#pragma unroll
      for (int q = 0; q < kHalf / 8; ++q)             // ncol is a multiple of 8
        ch[q].load(v + min(h0 + 8 * q, ncol - 8));   // past the end: a repeat, unused
      // (regions past R multiply unset LDS rows; their sums are never stored)
#pragma unroll
      for (int q = 0; q < kHalf / 8; ++q) {
        if (h0 + 8 * q < ncol) {
          double x[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) x[e] = ch[q].at(e);
#pragma unroll
          for (int r = 0; r < RM; ++r)
#pragma unroll
            for (int e = 0; e < 8; ++e) dot[r] = fma(x[e], cs[r][h0 + 8 * q + e], dot[r]);
        }
      }
    }
#pragma unroll
    for (int r = 0; r < RM; ++r)
      if (r < R) store_shared(&P[(size_t)i * a.r_max + r], dot[r]);   // read by the last slice
  }
  if (tid < 64) {
    // |c_r|^2 over the slice: lane l takes the columns l, l+64, ... in order,
    // then a fixed shuffle tree
    for (int r = 0; r < R; ++r) {
      double q = 0.0;
      for (int j = tid; j < ncol; j += 64) q = fma(cs[r][j], cs[r][j], q);
      q = wave_sum_f64(q);
      if (tid == 0) store_shared(&a.CN[((size_t)b * a.S + s) * a.r_max + r], q);
    }
  }
  if (tid < kRegMax) cnt[tid] = 0;
  if (!finish_and_check_last(&a.done[b], a.S, &last)) return;

  // ---- the question's last slice: assignment for the next step.  Rows in
  // blocks of 256: the (row, region) sums over the slices, four pairs and
  // eight slices of loads in flight per thread, in slice order; then one row
  // per thread takes its argmin.
  const double* Pb = a.P + (size_t)b * a.S * a.k_max * a.r_max;
  const double* CNb = a.CN + (size_t)b * a.S * a.r_max;
  __shared__ double cn[kRegMax];
  if (tid < R) {
    double q = 0.0;
    for (int z = 0; z < a.S; ++z) q += load_shared(&CNb[z * a.r_max + tid]);
    cn[tid] = q;
  }
  __syncthreads();
  const size_t zs = (size_t)a.k_max * a.r_max;      // one slice's partials
  for (int i0 = 0; i0 < k; i0 += kRegCols) {
    const int rows_here = min(kRegCols, k - i0);
    const int npair = rows_here * a.r_max;
    for (int f0 = tid; f0 < npair; f0 += kRegPairs * kRegCols) {
      double acc[kRegPairs];
      size_t off[kRegPairs];
      bool on[kRegPairs];
#pragma unroll
      for (int j = 0; j < kRegPairs; ++j) {
        const int f = f0 + j * kRegCols;
        on[j] = f < npair && (f % a.r_max) < R;
        off[j] = on[j] ? (size_t)i0 * a.r_max + f : 0;   // a valid slot when unused
        acc[j] = 0.0;
      }
      int z = 0;
      for (; z + 8 <= a.S; z += 8) {
        double x[8][kRegPairs];
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int j = 0; j < kRegPairs; ++j) x[u][j] = load_shared(&Pb[(size_t)(z + u) * zs + off[j]]);
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int j = 0; j < kRegPairs; ++j) acc[j] += x[u][j];
      }
      for (; z < a.S; ++z)
#pragma unroll
        for (int j = 0; j < kRegPairs; ++j) acc[j] += load_shared(&Pb[(size_t)z * zs + off[j]]);
#pragma unroll
      for (int j = 0; j < kRegPairs; ++j) {
        const int f = f0 + j * kRegCols;
        if (on[j]) dl[f] = cn[f % a.r_max] - 2.0 * acc[j];
      }
    }
    __syncthreads();
    if (tid < rows_here) {
      const int i = i0 + tid;
      int best = 0;
      double bd = dl[tid * a.r_max];
      for (int r = 1; r < R; ++r) {
        const double dist = dl[tid * a.r_max + r];
        if (dist < bd) {
          bd = dist;
          best = r;
        }
      }
      a.asg[k0 + i] = (uint8_t)best;
      asl[i] = (uint8_t)best;
      atomicAdd(&cnt[best], 1);
    }
    __syncthreads();
  }
  if (tid < R) a.sizes[b * a.r_max + tid] = cnt[tid];
  // row ids sorted by region, ascending within a region: region r starts at
  // the sizes of the smaller regions; a block scan per region and block of
  // 256 rows places each row after the earlier rows of its region
  __shared__ uint32_t scan_sh[kRegCols / 64 + 1];
  int base[RM];                                // next slot of each region (same in every thread)
  {
    int o = 0;
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      base[r] = o;
      if (r < R) o += cnt[r];
    }
  }
  for (int i0 = 0; i0 < k; i0 += kRegCols) {
    const int i = i0 + tid;
    const int ai = i < k ? (int)asl[i] : -1;
    const int id = i < k ? (int)row_id(i) : 0;
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      if (r < R) {
        uint32_t tot;
        const uint32_t pos = block_exclusive_scan(ai == r ? 1u : 0u, scan_sh, &tot);
        if (ai == r) {
          a.perm[k0 + base[r] + (int)pos] = id;
          a.sreg[k0 + base[r] + (int)pos] = (uint8_t)r;
        }
        base[r] += (int)tot;
      }
    }
  }
  if (tid == 0) a.done[b] = 0;
}

static size_t ralign(size_t n) { return (n + 255) & ~(size_t)255; }

int region_slices(const skip_problem_t& p) { return (p.d + kRegCols - 1) / kRegCols; }

size_t region_scratch_bytes(const skip_problem_t& p, int r_max) {
  const size_t S = (size_t)region_slices(p);
  return ralign((size_t)p.B * r_max * p.d * sizeof(double)) +
         ralign((size_t)p.B * S * p.k_max * r_max * sizeof(double)) +
         ralign((size_t)p.B * S * r_max * sizeof(double)) +
         ralign((size_t)p.total_kept) +
         ralign((size_t)p.total_kept * sizeof(int32_t)) +
         ralign((size_t)p.total_kept) +
         ralign((size_t)p.B * r_max * sizeof(int32_t)) +
         ralign((size_t)p.B * sizeof(int32_t));
}

template <typename T, bool IDX>
static void launch_step(int r_max, dim3 grid, dim3 block, hipStream_t s, const T* rows,
                        const RegionArgs& a) {
  if (r_max <= 4)
    hipLaunchKernelGGL((region_step_kernel<T, IDX, 4>), grid, block, 0, s, rows, a);
  else if (r_max <= 8)
    hipLaunchKernelGGL((region_step_kernel<T, IDX, 8>), grid, block, 0, s, rows, a);
  else
    hipLaunchKernelGGL((region_step_kernel<T, IDX, 16>), grid, block, 0, s, rows, a);
}

hipError_t launch_regions(const skip_problem_t& p, const void* rows, const int32_t* kept_offsets,
                          const int32_t* kept_idx, int r_max, int n_iter, int32_t* region,
                          float* centroids, int32_t* sizes, void* scratch, hipStream_t s) {
  const int S = region_slices(p);
  char* c = static_cast<char*>(scratch);
  RegionArgs a;
  a.kept_offsets = kept_offsets;
  a.kept_idx = kept_idx;
  a.N = p.N;
  a.total_kept = p.total_kept;
  a.B = p.B;
  a.d = p.d;
  a.k_max = p.k_max;
  a.r_max = r_max;
  a.S = S;
  a.n_iter = n_iter;
  a.C = reinterpret_cast<double*>(c);
  c += ralign((size_t)p.B * r_max * p.d * sizeof(double));
  a.P = reinterpret_cast<double*>(c);
  c += ralign((size_t)p.B * S * p.k_max * r_max * sizeof(double));
  a.CN = reinterpret_cast<double*>(c);
  c += ralign((size_t)p.B * S * r_max * sizeof(double));
  a.asg = reinterpret_cast<uint8_t*>(c);
  c += ralign((size_t)p.total_kept);
  a.perm = reinterpret_cast<int32_t*>(c);
  c += ralign((size_t)p.total_kept * sizeof(int32_t));
  a.sreg = reinterpret_cast<uint8_t*>(c);
  c += ralign((size_t)p.total_kept);
  a.sizes = reinterpret_cast<int32_t*>(c);
  c += ralign((size_t)p.B * r_max * sizeof(int32_t));
  a.done = reinterpret_cast<int32_t*>(c);
  a.region_out = region;
  a.cent_out = centroids;
  a.sizes_out = sizes;
  hipLaunchKernelGGL(region_clear_kernel, dim3(1), dim3(256), 0, s, a.done, p.B);
  const bool idx = kept_idx != nullptr;
  const dim3 grid(8 * ((p.B + 7) / 8) * S), block(kRegCols);
  for (int t = 0; t <= n_iter; ++t) {
    a.t = t;
    if (p.dtype == SKIP_F32) {
      if (idx) launch_step<float, true>(r_max, grid, block, s, (const float*)rows, a);
      else launch_step<float, false>(r_max, grid, block, s, (const float*)rows, a);
    } else {
      if (idx) launch_step<bf16_t, true>(r_max, grid, block, s, (const bf16_t*)rows, a);
      else launch_step<bf16_t, false>(r_max, grid, block, s, (const bf16_t*)rows, a);
    }
  }
  return hipGetLastError();
}

}  // namespace skip

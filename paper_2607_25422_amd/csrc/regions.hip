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
// order and assigns every row by argmin_r |c_r|^2 - 2 v_i . c_r, which is
// |v_i - c_r|^2 less the row's own |v_i|^2.
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

// 16 bytes of a row held in LDS: 8 bf16 or 4 f32 elements, as doubles
template <typename T> struct RegLds;
template <> struct RegLds<bf16_t> {
  static constexpr int n = 8;
  u32x4 w;
  __device__ __forceinline__ void load(const uint8_t* p) { w = *reinterpret_cast<const u32x4*>(p); }
  __device__ __forceinline__ double at(int e) const {
    const uint32_t x = w[e >> 1];
    return (double)__uint_as_float((e & 1) ? (x & 0xffff0000u) : (x << 16));
  }
};
template <> struct RegLds<float> {
  static constexpr int n = 4;
  u32x4 w;
  __device__ __forceinline__ void load(const uint8_t* p) { w = *reinterpret_cast<const u32x4*>(p); }
  __device__ __forceinline__ double at(int e) const { return (double)__uint_as_float(w[e]); }
};

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
  double* P;                   // [B][S][r_max][k_max + 1] partial v_i . c_r, then |c_r|^2
  int PK;                      // k_max + 1: the region stride of P
  uint8_t* asg;                // [total_kept]        current assignment
  int32_t* perm;               // [total_kept]        positions in the question sorted by region (stable)
  uint8_t* sreg;               // [total_kept]        region of each sorted position
  int32_t* sizes;              // [B][r_max]          rows per region
  int32_t* done;               // [B]                 finished slices
  int32_t* region_out;         // [total_kept]
  float* cent_out;             // [B][r_max][d]
  int32_t* sizes_out;          // [B][r_max] or NULL
};

constexpr int kRegRowBatch = 32;   // rows whose loads are issued together (update)
constexpr int kRegPairs = 8;       // (row, region) sums per thread at once (assignment)
constexpr int kRegBufferFlags = 0x00020000;   // buffer resource word 3 (gfx9 raw buffer)
constexpr int kRegSc1 = 16;                   // buffer load cache policy: sc1

// Rows per lane in a block of rows of the dot products (each lane's share of
// a centroid value read from LDS); the block is staged whole in LDS.
template <int RM> struct RegDotRows { static constexpr int n = RM > 8 ? 2 : 3; };
// LDS shared by the phases: per wave a block of up to 3 x 64 rows of 128
// bytes and one zero row
constexpr int kRegPoolBytes = 4 * (3 * 64 + 1) * 128;
constexpr int kRegIds = 8192;                       // sorted rows staged at once (update)
constexpr int kRegResidentRows = 3 * 64;            // largest resident block (RPL = 3)
constexpr int kRegUpdBatch = 16;                     // resident values read at once (update)

// RM: a compile-time bound on the regions (4, 8 or 16), so that every loop
// over the regions unrolls and the per-region sums stay in fixed registers
// (a run-time bound made the compiler index the register file, one
// instruction at a time).
template <typename T, bool IDX, int RM>
__global__ void __launch_bounds__(kRegCols)
region_step_kernel(const T* __restrict__ rows, RegionArgs a) {
  __shared__ __align__(16) double cs[kRegMax][kRegCols];    // this step's centroids, this slice
  // One pool, carved per phase:
  //   update       row ids [kRegIds] int32, then their regions [kRegIds] uint8
  //   dots         the block of rows, per wave [RPL * 64][128 bytes], later
  //                the sums of waves 1-3 [3][RPL * RM][64] double
  //   last slice   distances [256][16] double, then the assignment [k] uint8
  __shared__ __align__(16) uint8_t pool[kRegPoolBytes];
  static_assert(kRegIds * 5 <= kRegPoolBytes, "update staging fits the pool");
  static_assert(kRegCols * kRegMax * 8 + kRegMaxRows <= kRegPoolBytes, "assignment fits the pool");
  __shared__ int last;
  __shared__ int cnt[kRegMax];
  // LDS addresses of the sorted positions, when the rows are resident
  __shared__ __align__(16) int spos[kRegResidentRows + (kRegMax + 1) * kRegUpdBatch];
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

  // ---- rows of the question in LDS.  Wave w holds the slice's columns
  // [64w, 64w + 64) of a block of 64 RPL rows, 128 bytes of a row per pass
  // (64 bf16 or 32 f32 columns), copied with direct loads: eight lanes fetch
  // one row's line, so every load instruction reads whole lines.  Chunk q of
  // local row j sits at slot q ^ (j & 7) of the row's 128 bytes, so that the
  // lanes' reads of one chunk of their own rows fall on distinct LDS banks.
  // When a bf16 question fits one block its rows stay resident for the whole
  // step: loaded once here, read by the centroid update and the products.
  constexpr int RPL = RegDotRows<RM>::n;
  constexpr int EPC = RegLds<T>::n;                // columns per 16-byte chunk
  constexpr int NP = 64 / (8 * EPC);               // passes over the wave's columns
  constexpr int WROWS = RPL * 64 + 1;              // rows of a wave's block, the last one zero
  static_assert(4 * WROWS * 128 <= kRegPoolBytes, "row block fits the pool");
  static_assert(64 * RPL <= kRegResidentRows, "resident positions fit");
  const int w = tid >> 6, lane = tid & 63;
  uint8_t* wrows = pool + w * (WROWS * 128);        // this wave's rows
  const uint32_t wlds = lds_addr(wrows);
  const bool resident = NP == 1 && k <= 64 * RPL;
  auto stage_rows = [&](int blk0, int pass) {
    // lane l fetches chunk (l & 7) ^ (l >> 3) of local row 8j + (l >> 3);
    // rows past the question repeat its last row, columns past the slice its
    // first chunk (their centroid values are 0).  The row indices are all
    // read before the first copy: the copies are opaque to the compiler,
    // which would otherwise wait for each one before the next index.
    const int q = (lane & 7) ^ (lane >> 3);
    const int col = 64 * w + pass * 8 * EPC + q * EPC;
    const int colc = col < ncol ? col : 0;
    int rid[8 * RPL];
#pragma unroll
    for (int j = 0; j < 8 * RPL; ++j) {
      const int i = min(blk0 + 8 * j + (lane >> 3), k - 1);
      rid[j] = IDX ? a.kept_idx[k0 + i] : k0 + i;
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < 8 * RPL; ++j) {
      const size_t row = IDX ? (size_t)b * a.N + clampi(rid[j], 0, a.N - 1) : (size_t)rid[j];
      lds_dma16(rows + row * a.d + c0 + colc, wlds + j * 1024);
    }
  };
  // element (local row lr, slice column tid) of a resident block
  auto resident_at = [&](int lr) -> double {
    const uint8_t* e = wrows + lr * 128 + (((lane >> 3) ^ (lr & 7)) * 16) + (lane & 7) * sizeof(T);
    return reg_load1<T>(reinterpret_cast<const T*>(e));
  };
  if (resident) stage_rows(0, 0);

  // ---- centroids of this step, this slice's columns (thread = column)
  if (a.t == 0) {
    if (resident) wait_vmcnt<0>();                  // a wave reads only rows it copied
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      if (r < R) {
        const int pos = ((2 * r + 1) * k) / (2 * R);
        cs[r][tid] = cok ? (resident ? resident_at(pos) : reg_load1<T>(row_of(pos) + c)) : 0.0;
      }
    }
  } else {
    // the rows sorted by region (perm: positions in the question, ascending
    // within a region; sreg: the region of each sorted position) are summed
    // in one pass: each thread keeps its column's running sum in a register
    // and hands it to LDS where the region changes (a uniform test).  32
    // values are read together, positions and columns clamped into range
    // (padding repeats the last position, marked region 0xff: skipped).
    // Regions without rows keep their centroid.
    for (int r = tid; r < R; r += blockDim.x) cnt[r] = a.sizes[b * a.r_max + r];
    const int cc = cok ? c : c0;
    int cur = -1;
    double acc = 0.0;
    auto take = [&](const double (&v)[kRegRowBatch], const uint32_t (&rg4)[kRegRowBatch / 4]) {
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
    };
    if (resident) {
      // Region by region (sizes give the runs of the sorted order), sixteen
      // values at a time into four running sums (value u of a batch into sum
      // u % 4; the sums are added pairwise at the end of the region).  The
      // staged words give the lane-independent part of each value's LDS
      // address, 128 lr + 16 (lr & 7) for row lr: the lane's element is then
      // at (word ^ 16 (l >> 3)) + 2 (l & 7) past the wave's rows.  Each run is
      // padded to a whole batch with the word of the wave's zero row, and the
      // next batch's words are read before the current batch's values.
      uint32_t* zrow = reinterpret_cast<uint32_t*>(wrows + (WROWS - 1) * 128);
      if (lane < 32) zrow[lane] = 0u;
      const int zword = (WROWS - 1) * 128;         // (WROWS - 1) is a multiple of 8
      __syncthreads();                             // cnt
      int pst[RM], rst[RM], np_all = 0;
      {
        int o = 0;
#pragma unroll
        for (int r = 0; r < RM; ++r) {
          const int n = r < R ? cnt[r] : 0;
          pst[r] = np_all;
          rst[r] = o;
          np_all += (n + kRegUpdBatch - 1) / kRegUpdBatch * kRegUpdBatch;
          o += n;
        }
      }
      for (int p = tid; p < np_all + kRegUpdBatch; p += blockDim.x) {
        int r = 0;
#pragma unroll
        for (int q = 1; q < RM; ++q)
          if (q < R && p >= pst[q]) r = q;
        const int i = p - pst[r];
        int word = zword;
        if (p < np_all && i < cnt[r]) {
          const int lr = clampi(a.perm[k0 + rst[r] + i], 0, k - 1);
          word = lr * 128 + ((lr & 7) << 4);
        }
        spos[p] = word;
      }
      wait_vmcnt<0>();
      __syncthreads();
      const uint32_t lsw = (uint32_t)((lane >> 3) << 4);
      const uint8_t* wl = wrows + (lane & 7) * sizeof(T);
      int pwn[kRegUpdBatch];
#pragma unroll
      for (int u = 0; u < kRegUpdBatch; ++u) pwn[u] = spos[u];
#pragma unroll
      for (int r = 0; r < RM; ++r) {
        if (r < R) {
          const int n = cnt[r];
          const int np = (n + kRegUpdBatch - 1) / kRegUpdBatch * kRegUpdBatch;
          double racc[4] = {0.0, 0.0, 0.0, 0.0};
          for (int j0 = 0; j0 < np; j0 += kRegUpdBatch) {
            int pw[kRegUpdBatch];
#pragma unroll
            for (int u = 0; u < kRegUpdBatch; ++u) {
              pw[u] = pwn[u];
              pwn[u] = spos[pst[r] + j0 + kRegUpdBatch + u];
            }
            double v[kRegUpdBatch];
#pragma unroll
            for (int u = 0; u < kRegUpdBatch; ++u)
              v[u] = reg_load1<T>(reinterpret_cast<const T*>(wl + (((uint32_t)pw[u]) ^ lsw)));
#pragma unroll
            for (int u = 0; u < kRegUpdBatch; ++u) racc[u & 3] += v[u];
          }
          if (n > 0) cs[r][tid] = (racc[0] + racc[1]) + (racc[2] + racc[3]);
        }
      }
    } else {
      // row indices and regions staged in LDS 8192 at a time
      int* ids = reinterpret_cast<int*>(pool);
      uint8_t* srg = pool + kRegIds * sizeof(int);
      constexpr int kIds = kRegIds;
      for (int g0 = 0; g0 < k; g0 += kIds) {
        const int ng = min(kIds, k - g0);
        const int ng32 = (ng + kRegRowBatch - 1) / kRegRowBatch * kRegRowBatch;
        __syncthreads();                 // the previous group is consumed
        for (int j = tid; j < ng32; j += blockDim.x) {
          const int jj = min(j, ng - 1);
          ids[j] = (int)row_id(clampi(a.perm[k0 + g0 + jj], 0, k - 1));
          srg[j] = (j < ng) ? a.sreg[k0 + g0 + jj] : (uint8_t)0xff;
        }
        __syncthreads();
        for (int j0 = 0; j0 < ng; j0 += kRegRowBatch) {
          double v[kRegRowBatch];
          int4 id4[kRegRowBatch / 4];
          uint32_t rg4[kRegRowBatch / 4];
#pragma unroll
          for (int q = 0; q < kRegRowBatch / 4; ++q) {
            id4[q] = *reinterpret_cast<const int4*>(&ids[j0 + 4 * q]);
            rg4[q] = *reinterpret_cast<const uint32_t*>(&srg[j0 + 4 * q]);
          }
#pragma unroll
          for (int q = 0; q < kRegRowBatch / 4; ++q) {
            v[4 * q + 0] = reg_load1<T>(rows + (size_t)id4[q].x * a.d + cc);
            v[4 * q + 1] = reg_load1<T>(rows + (size_t)id4[q].y * a.d + cc);
            v[4 * q + 2] = reg_load1<T>(rows + (size_t)id4[q].z * a.d + cc);
            v[4 * q + 3] = reg_load1<T>(rows + (size_t)id4[q].w * a.d + cc);
          }
          __builtin_amdgcn_sched_barrier(0);
          take(v, rg4);
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

  // ---- partial products over this slice.  Wave w takes the slice's columns
  // [64w, 64w + 64) and lane l the rows l, l + 64, ... of a block of rows
  // (RPL rows per lane, staged in LDS as described above), so that each
  // centroid value read from LDS (one address for the whole wave) feeds RPL
  // rows.  Waves 1-3 then hand their sums to wave 0 through LDS, which adds
  // them in wave order and stores them.
  constexpr int NV = RPL * RM;
  static_assert(3 * NV * 64 * (int)sizeof(double) <= kRegPoolBytes, "wave sums fit the pool");
  double* P = a.P + ((size_t)b * a.S + s) * a.PK * a.r_max;
  double* red = reinterpret_cast<double*>(pool);   // [3][NV][64] sums of waves 1-3
  for (int blk0 = 0; blk0 < k; blk0 += 64 * RPL) {
    double dot[RPL][RM];
#pragma unroll
    for (int rr = 0; rr < RPL; ++rr)
#pragma unroll
      for (int r = 0; r < RM; ++r) dot[rr][r] = 0.0;
#pragma unroll
    for (int pass = 0; pass < NP; ++pass) {
      if (!resident) {
        stage_rows(blk0, pass);
        wait_vmcnt<0>();
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        RegLds<T> x[RPL];
#pragma unroll
        for (int rr = 0; rr < RPL; ++rr)
          x[rr].load(wrows + (rr * 64 + lane) * 128 + ((q ^ (lane & 7)) * 16));
        const int col = 64 * w + pass * 8 * EPC + q * EPC;
#pragma unroll
        for (int e = 0; e < EPC; ++e) {
          double xv[RPL];
#pragma unroll
          for (int rr = 0; rr < RPL; ++rr) xv[rr] = x[rr].at(e);
          // (regions past R multiply unset LDS rows; their sums are never stored)
#pragma unroll
          for (int r = 0; r < RM; ++r) {
            const double cv = cs[r][col + e];
#pragma unroll
            for (int rr = 0; rr < RPL; ++rr) dot[rr][r] = fma(xv[rr], cv, dot[rr][r]);
          }
        }
      }
      asm volatile("" ::: "memory");      // the reads above precede the next pass's loads
      __builtin_amdgcn_s_waitcnt(0xC07F); // lgkmcnt(0)
    }
    __syncthreads();                      // every wave is done with its rows
    if (w > 0) {
#pragma unroll
      for (int v = 0; v < NV; ++v) red[((w - 1) * NV + v) * 64 + lane] = dot[v / RM][v % RM];
    }
    __syncthreads();
    if (w == 0) {
#pragma unroll
      for (int rr = 0; rr < RPL; ++rr) {
        const int i = blk0 + rr * 64 + lane;
#pragma unroll
        for (int r = 0; r < RM; ++r) {
          const int v = rr * RM + r;
          const double sum = ((dot[rr][r] + red[v * 64 + lane]) + red[(NV + v) * 64 + lane]) +
                             red[(2 * NV + v) * 64 + lane];
          if (r < R && i < k) store_shared(&P[(size_t)r * a.PK + i], sum);   // read by the last slice
        }
      }
    }
    __syncthreads();                      // the sums are read before the pool is reused
  }
  {
    // |c_r|^2 over the slice: wave w takes the regions w, w + 4, ..., lane l
    // the columns l, l + 64, l + 128, l + 192 in order (columns past the
    // slice hold 0), then a fixed shuffle tree over all of the wave's regions
    // at once
    constexpr int RW = (RM + 3) / 4;
    double q[RW];
#pragma unroll
    for (int u = 0; u < RW; ++u) {
      const int r = min(w + 4 * u, RM - 1);
      q[u] = 0.0;
#pragma unroll
      for (int j = 0; j < kRegCols / 64; ++j) q[u] = fma(cs[r][lane + 64 * j], cs[r][lane + 64 * j], q[u]);
    }
#pragma unroll
    for (int sh = 32; sh >= 1; sh >>= 1)
#pragma unroll
      for (int u = 0; u < RW; ++u) q[u] += __shfl_xor(q[u], sh, kWave);
    if (lane == 0) {
#pragma unroll
      for (int u = 0; u < RW; ++u)
        if (w + 4 * u < R) store_shared(&P[(size_t)(w + 4 * u) * a.PK + a.k_max], q[u]);
    }
  }
  if (tid < kRegMax) cnt[tid] = 0;
  if (!finish_and_check_last(&a.done[b], a.S, &last)) return;

  // ---- the question's last slice: assignment for the next step.  Rows in
  // blocks of 256: the (row, region) sums over the slices, with the regions'
  // |c_r|^2 as R more pairs of the first block, eight pairs and eight slices
  // of loads in flight per thread, in slice order; then one row per thread
  // takes its argmin, and each wave counts its rows per region.
  double* dl = reinterpret_cast<double*>(pool);                 // [256][r_max] v_i . c_r
  uint8_t* asl = pool + kRegCols * kRegMax * sizeof(double);    // [k]
  const double* Pb = a.P + (size_t)b * a.S * a.PK * a.r_max;
  __shared__ double cn[kRegMax];
  __shared__ int cw[kRegCols / 64][kRegMax];
  const size_t zs = (size_t)a.PK * a.r_max;         // one slice's partials
  const auto prsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<double*>(Pb), 0, (int)(a.S * zs * sizeof(double)), kRegBufferFlags);
  for (int i0 = 0; i0 < k; i0 += kRegCols) {
    const int rows_here = min(kRegCols, k - i0);
    const int nrow_pairs = rows_here * R;
    const int npair = nrow_pairs + (i0 == 0 ? R : 0);
    for (int f0 = tid; f0 < npair; f0 += kRegPairs * kRegCols) {
      // pair f < nrow_pairs: (region f / rows_here, row f % rows_here of the
      // block); past them: |c_r|^2 of region f - nrow_pairs
      double acc[kRegPairs];
      uint32_t off[kRegPairs];
#pragma unroll
      for (int j = 0; j < kRegPairs; ++j) {
        const int f = min(f0 + j * kRegCols, npair - 1);        // past the end: a repeat, unused
        int slot;
        if (f < nrow_pairs) {
          const int r = f / rows_here;
          slot = r * a.PK + i0 + (f - r * rows_here);
        } else {
          slot = (f - nrow_pairs) * a.PK + a.k_max;
        }
        off[j] = (uint32_t)slot * (uint32_t)sizeof(double);
        acc[j] = 0.0;
      }
      // Buffer loads: the question's partials as one resource, the slice as
      // a scalar offset, the pair as a 32-bit byte offset (a 64-bit address
      // per load would take two registers each).  Cache policy sc1, as for
      // the other reads of values the slices published.
      auto part = [&](int z, int j) -> double {
        const auto v = __builtin_amdgcn_raw_buffer_load_b64(
            prsrc, off[j], (int)((size_t)z * zs * sizeof(double)), kRegSc1);
        return __builtin_bit_cast(double, v);
      };
      int z = 0;
      for (; z + 8 <= a.S; z += 8) {
        double x[8][kRegPairs];
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int j = 0; j < kRegPairs; ++j) x[u][j] = part(z + u, j);
#pragma unroll
        for (int u = 0; u < 8; ++u)
#pragma unroll
          for (int j = 0; j < kRegPairs; ++j) acc[j] += x[u][j];
      }
      for (; z < a.S; ++z)
#pragma unroll
        for (int j = 0; j < kRegPairs; ++j) acc[j] += part(z, j);
#pragma unroll
      for (int j = 0; j < kRegPairs; ++j) {
        const int f = f0 + j * kRegCols;
        if (f < nrow_pairs) {
          const int r = f / rows_here;
          dl[(f - r * rows_here) * a.r_max + r] = acc[j];
        } else if (f < npair) {
          cn[f - nrow_pairs] = acc[j];
        }
      }
    }
    __syncthreads();
    int best = -1;
    if (tid < rows_here) {
      const int i = i0 + tid;
      best = 0;
      double bd = cn[0] - 2.0 * dl[tid * a.r_max];
      for (int r = 1; r < R; ++r) {
        const double dist = cn[r] - 2.0 * dl[tid * a.r_max + r];
        if (dist < bd) {
          bd = dist;
          best = r;
        }
      }
      a.asg[k0 + i] = (uint8_t)best;
      asl[i] = (uint8_t)best;
    }
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      if (r < R) {
        const uint64_t m = __ballot(best == r);
        if (lane == 0 && m != 0) atomicAdd(&cnt[r], (int)__popcll(m));
      }
    }
    __syncthreads();
  }
  if (tid < R) a.sizes[b * a.r_max + tid] = cnt[tid];
  // row ids sorted by region, ascending within a region: region r starts at
  // the sizes of the smaller regions; within a block of 256 rows a row goes
  // after the block's earlier rows of its region (the counts of the earlier
  // waves, then the lanes below it in its wave's ballot)
  int base[RM];                                // next slot of each region (same in every thread)
  {
    int o = 0;
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      base[r] = o;
      if (r < R) o += cnt[r];
    }
  }
  const uint64_t below = (1ull << lane) - 1ull;
  for (int i0 = 0; i0 < k; i0 += kRegCols) {
    const int i = i0 + tid;
    const int ai = i < k ? (int)asl[i] : -1;
    uint64_t mine = 0;
    int off = 0;
#pragma unroll
    for (int r = 0; r < RM; ++r) {
      if (r < R) {
        const uint64_t m = __ballot(ai == r);
        if (lane == 0) cw[w][r] = (int)__popcll(m);
        if (ai == r) {
          mine = m;
          off = base[r];
        }
      }
    }
    __syncthreads();
    if (ai >= 0) {
      for (int v = 0; v < w; ++v) off += cw[v][ai];
      off += (int)__popcll(mine & below);
      a.perm[k0 + off] = i;
      a.sreg[k0 + off] = (uint8_t)ai;
    }
#pragma unroll
    for (int r = 0; r < RM; ++r)
      if (r < R) base[r] += cw[0][r] + cw[1][r] + cw[2][r] + cw[3][r];
    __syncthreads();                             // the counts are reused
  }
  if (tid == 0) a.done[b] = 0;
}

static size_t ralign(size_t n) { return (n + 255) & ~(size_t)255; }

int region_slices(const skip_problem_t& p) { return (p.d + kRegCols - 1) / kRegCols; }

size_t region_scratch_bytes(const skip_problem_t& p, int r_max) {
  const size_t S = (size_t)region_slices(p);
  return ralign((size_t)p.B * r_max * p.d * sizeof(double)) +
         ralign((size_t)p.B * S * (p.k_max + 1) * r_max * sizeof(double)) +
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
  a.PK = p.k_max + 1;
  c += ralign((size_t)p.B * S * (p.k_max + 1) * r_max * sizeof(double));
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

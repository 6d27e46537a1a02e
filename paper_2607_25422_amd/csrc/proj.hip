// Learned projection of the kept rows (paper eq. bsca: W_v v_i and W_k k_j
// before their inner product; Def. B.3: h_v, h_k; the attention query W_Q v):
//
//   Y[r] = W x_r,   x_r the kept row r (given rows, or V[b][kept_idx[r]]),
//   W: [d_out][d] bf16, float32 sums on v_mfma_f32_32x32x16_bf16.
//
//   proj_pack_kernel : W repacked in the order the GEMM's waves read it (one
//                      1 KiB run per wave, step and k16 sub-step)
//   proj_gemm_kernel : work item = (128 kept rows, 256 output columns); the
//                      row tile arrives in a 4-slot LDS ring by direct
//                      global->LDS loads three 32-column steps ahead, rows
//                      gathered through kept_idx as they are loaded; each
//                      wave's weight fragments come straight from the packed
//                      copy into registers two steps ahead; 8 waves of 32
//                      output columns x 96 rows (3 blocks of 32 x 32)
#include <algorithm>

#include "skip_common.h"
#include "skip_internal.h"

namespace skip {

// rows per tile: 3 blocks of 32 (3072 kept rows make 32 tiles, so with 16
// column tiles 512 items fill 256 CUs twice over)
constexpr int kProjMT = 96;
constexpr int kProjMB = kProjMT / 32;     // 32-row blocks per tile
constexpr int kProjNT = 256;       // output columns per tile (8 waves x 32)
constexpr int kProjKS = 32;        // columns of d per step
constexpr int kProjThreads = 512;
constexpr int kProjRing = 4;
constexpr int kProjAhead = 3;
constexpr int kProjPackBlocks = 1024;

// Packed order: for column tile nt, wave w, step s, k16 sub-step kk and lane
// l, the 16 bytes W[256 nt + 32 w + l % 32][32 s + 8 (2 kk + l / 32) .. +7].
__global__ void __launch_bounds__(256)
proj_pack_kernel(const bf16_t* __restrict__ W, int d, int d_out, u32x4* __restrict__ Wp) {
  const size_t total = (size_t)d_out * d / 8;          // 16-byte units
  const int ksteps = d / kProjKS;
  for (size_t u = (size_t)blockIdx.x * blockDim.x + threadIdx.x; u < total;
       u += (size_t)gridDim.x * blockDim.x) {
    const int l = (int)(u % 64);
    size_t r = u / 64;
    const int kk = (int)(r % 2); r /= 2;
    const int s = (int)(r % ksteps); r /= ksteps;
    const int w = (int)(r % 8);
    const int nt = (int)(r / 8);
    const int j = nt * kProjNT + w * 32 + (l & 31);
    const int col = s * kProjKS + (2 * kk + (l >> 5)) * 8;
    Wp[u] = *reinterpret_cast<const u32x4*>(W + (size_t)j * d + col);
  }
}

// Work items are dealt to XCDs in runs (the hardware sends workgroup id L to
// XCD L % 8): item = (L % 8) * per_xcd + L / 8, row tile fastest, so the
// items of one XCD share their weight tiles in its L2.
template <bool IDX, bool OUT_F32>
__global__ void __launch_bounds__(kProjThreads)
proj_gemm_kernel(const bf16_t* __restrict__ rows, const int32_t* __restrict__ kept_offsets,
                 const int32_t* __restrict__ kept_idx, int B, int N, int M, int d, int d_out,
                 const u32x4* __restrict__ Wp, void* __restrict__ Y, int n_items) {
  constexpr int A_ELEMS = kProjMT * kProjKS;          // 3072 (6 KiB)
  __shared__ __attribute__((aligned(1024))) bf16_t Ar[kProjRing * A_ELEMS];

  const int per_xcd = gridDim.x / 8;
  const int item = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (item >= n_items) return;
  const int MTL = (M + kProjMT - 1) / kProjMT;
  const int mt = item % MTL, nt = item / MTL;
  const int i0 = mt * kProjMT, j0 = nt * kProjNT;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ksteps = d / kProjKS;
  const int hh = lane >> 5, r32 = lane & 31;

  // this thread's 16 bytes of a row tile: row tid/4 of the tile, physical
  // chunk tid%4 holding logical chunk lc (XOR-swizzled by (row/2) % 4, so the
  // operand reads of 8 consecutive rows hit distinct banks)
  const int trow = tid >> 2;
  const int lc = (tid & 3) ^ ((trow >> 1) & 3);
  const int r = min(i0 + trow, M - 1);
  size_t rid = (size_t)r;
  if (IDX) {
    // question of kept row r (kept_offsets ascending), then its row of V
    int lo = 0, hi = B;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (clampi(kept_offsets[mid], 0, M) <= r) lo = mid;
      else hi = mid;
    }
    rid = (size_t)lo * N + clampi(kept_idx[r], 0, N - 1);
  }
  const bf16_t* asrc = rows + rid * d + lc * 8;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t ar_lds = lds_addr(Ar) + (uint32_t)(wave_s * 1024);
  // (waves past the tile's rows, 4 * kProjMT threads and up, copy nothing)
  const bool a_loader = tid < 4 * kProjMT;
  auto issue_a = [&](int s) {
    if (a_loader)
      lds_dma16(asrc + s * kProjKS, __builtin_amdgcn_readfirstlane(
                                     ar_lds + (uint32_t)((s % kProjRing) * A_ELEMS * 2)));
  };
  const u32x4* wsrc = Wp + ((size_t)(nt * 8 + wave) * ksteps) * 128 + lane;
  auto load_w = [&](int s, u32x4 (&w)[2]) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) w[kk] = wsrc[(size_t)s * 128 + kk * 64];
  };

  f32x16_t acc[kProjMB];
#pragma unroll
  for (int mb = 0; mb < kProjMB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[mb][v] = 0.f;

  int aoff[2][kProjMB];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int mb = 0; mb < kProjMB; ++mb) {
      const int row = mb * 32 + r32;
      aoff[kk][mb] = row * kProjKS + (((2 * kk + hh) ^ ((row >> 1) & 3)) << 3);
    }

  auto mma_step = [&](int s, const u32x4 (&w)[2]) {
    __builtin_amdgcn_sched_barrier(0);
    const bf16_t* At = Ar + (s % kProjRing) * A_ELEMS;
    u32x4 a[2][kProjMB];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int mb = 0; mb < kProjMB; ++mb) a[kk][mb] = *reinterpret_cast<const u32x4*>(At + aoff[kk][mb]);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int mb = 0; mb < kProjMB; ++mb) acc[mb] = mfma32_bf16(a[kk][mb], w[kk], acc[mb]);
    // half the operand reads ahead, then one MFMA per read
    constexpr int NR = 2 * kProjMB;          // operand reads (= MFMAs)
    __builtin_amdgcn_sched_group_barrier(0x100, NR / 2, 0);
#pragma unroll
    for (int i = 0; i < NR / 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, NR / 2, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

#pragma unroll
  for (int a = 0; a < kProjAhead; ++a)
    if (a < ksteps) issue_a(a);
  u32x4 wA[2], wB[2];
  load_w(0, wA);
  load_w(min(1, ksteps - 1), wB);

  // Step s: wait for the row tile of step s (outstanding after the wait: the
  // tiles of steps s+1, s+2 while they exist, and the fragments of step s+1),
  // barrier (publishes it; the slot of step s-1 is free), load the tile of
  // step s+3, multiply step s, load the fragments of step s+2.
  auto step = [&](int s, u32x4 (&w)[2]) {
    if (s + 2 < ksteps) wait_vmcnt<4>();
    else if (s + 1 < ksteps) wait_vmcnt<3>();
    else wait_vmcnt<2>();
    barrier_nofence();
    if (s + kProjAhead < ksteps) issue_a(s + kProjAhead);
    mma_step(s, w);
    // unconditional (the last steps reload the final fragments): a
    // conditional load would make the compiler drain the queue before the
    // next use of w
    load_w(min(s + 2, ksteps - 1), w);
  };
  int s = 0;
  for (; s + 1 < ksteps; s += 2) {
    step(s, wA);
    step(s + 1, wB);
  }
  if (s < ksteps) step(s, wA);

  // Accumulator element v of block mb: row mb*32 + 8*(v/4) + 4*hh + v%4,
  // column j0 + 32*wave + r32.
  const int j = j0 + wave * 32 + r32;
#pragma unroll
  for (int mb = 0; mb < kProjMB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int row = i0 + mb * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
      if (row < M) {
        if (OUT_F32)
          static_cast<float*>(Y)[(size_t)row * d_out + j] = acc[mb][v];
        else
          static_cast<bf16_t*>(Y)[(size_t)row * d_out + j] = (bf16_t)f32_to_bf16(acc[mb][v]);
      }
    }
}

size_t proj_scratch_bytes(int d, int d_out) {
  return ((size_t)d_out * d * sizeof(bf16_t) + 255) & ~(size_t)255;
}

hipError_t launch_proj_pack(int d, int d_out, const void* W, void* packed, hipStream_t s) {
  hipLaunchKernelGGL(proj_pack_kernel, dim3(kProjPackBlocks), dim3(256), 0, s,
                     (const bf16_t*)W, d, d_out, static_cast<u32x4*>(packed));
  return hipGetLastError();
}

hipError_t launch_proj_gemm(const skip_problem_t& p, const void* rows, const int32_t* kept_offsets,
                            const int32_t* kept_idx, const void* packed, int d_out, void* Y,
                            int out_f32, hipStream_t s) {
  const int M = p.total_kept;
  if (M <= 0) return hipSuccess;
  const int n_items = ((M + kProjMT - 1) / kProjMT) * (d_out / kProjNT);
  const int grid = ((n_items + 7) / 8) * 8;
  const bf16_t* R = static_cast<const bf16_t*>(rows);
  const u32x4* Wc = static_cast<const u32x4*>(packed);
  if (kept_idx) {
    if (out_f32)
      hipLaunchKernelGGL((proj_gemm_kernel<true, true>), dim3(grid), dim3(kProjThreads), 0, s,
                         R, kept_offsets, kept_idx, p.B, p.N, M, p.d, d_out, Wc, Y, n_items);
    else
      hipLaunchKernelGGL((proj_gemm_kernel<true, false>), dim3(grid), dim3(kProjThreads), 0, s,
                         R, kept_offsets, kept_idx, p.B, p.N, M, p.d, d_out, Wc, Y, n_items);
  } else {
    if (out_f32)
      hipLaunchKernelGGL((proj_gemm_kernel<false, true>), dim3(grid), dim3(kProjThreads), 0, s,
                         R, kept_offsets, kept_idx, p.B, p.N, M, p.d, d_out, Wc, Y, n_items);
    else
      hipLaunchKernelGGL((proj_gemm_kernel<false, false>), dim3(grid), dim3(kProjThreads), 0, s,
                         R, kept_offsets, kept_idx, p.B, p.N, M, p.d, d_out, Wc, Y, n_items);
  }
  return hipGetLastError();
}

// Passage keys as bf16 rows for the projection: k~ = the bf16 rounding
// (through float, nearest even at both steps) of the pooled double key or of
// the caller's float key.
__global__ void __launch_bounds__(256)
keys_bf16_kernel(const double* __restrict__ kbar, const float* __restrict__ given, size_t n,
                 bf16_t* __restrict__ out) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x) {
    const float f = given ? given[i] : (float)kbar[i];
    out[i] = __builtin_bit_cast(bf16_t, (__bf16)f);
  }
}

hipError_t launch_keys_bf16(const double* kbar, const float* given, size_t n, void* out,
                            hipStream_t s) {
  if (n == 0) return hipSuccess;
  const size_t blocks = std::min<size_t>((n + 255) / 256, 4096);
  hipLaunchKernelGGL(keys_bf16_kernel, dim3((unsigned)blocks), dim3(256), 0, s, kbar, given, n,
                     static_cast<bf16_t*>(out));
  return hipGetLastError();
}

hipError_t launch_project(const skip_problem_t& p, const void* rows, const int32_t* kept_offsets,
                          const int32_t* kept_idx, const void* W, int d_out, void* Y,
                          int out_f32, void* scratch, hipStream_t s) {
  if (p.total_kept <= 0) return hipSuccess;
  hipError_t e = launch_proj_pack(p.d, d_out, W, scratch, s);
  if (e != hipSuccess) return e;
  return launch_proj_gemm(p, rows, kept_offsets, kept_idx, scratch, d_out, Y, out_f32, s);
}

}  // namespace skip

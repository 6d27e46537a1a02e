// Main-text salience scorer (paper Sec. 3.3, eq. qvs): a two-layer
// perceptron on the concatenation [v_i ; q_bar ; v_i * q_bar],
//
//   a_i = W1 x_i + b1,   s_i = w2 . relu(a_i) + b2,   W1: [h][3d] bf16.
//
// The model runs in bf16: q_bar enters rounded to bf16 (through float32) and
// the Hadamard term is the bf16 rounding of the exact product of two bf16
// values.  Split by where the work is:
//   mlp_prep_kernel  : q_bar' = bf16(q_bar) per question and the per-question
//                      constant c_b = W1[:, d:2d] q_bar' + b1 (float32 sums of
//                      exact products)
//   mlp_score_kernel : per question the GEMM [v_i | bf16(v_i * q_bar')] x
//                      [W1[:, 0:d] | W1[:, 2d:3d]]^T on v_mfma_f32_32x32x16_bf16
//                      (the Hadamard operand is formed in registers from the
//                      staged v tile), with relu(. + c_b) . w2 folded into the
//                      epilogue: one float partial of s_i per 256 hidden units
//   mlp_sum_kernel   : s_i = sum of the partials (fixed order) + b2, as the
//                      float64 ranking key of the top-k and as the output score
#include "skip_common.h"
#include "skip_internal.h"

namespace skip {

namespace {

// bf16(a * q) for the 8 bf16 values of a (q: 8 floats); a product of two
// bf16 values is exact in float32, so the pair conversion (round to nearest
// even, v_cvt_pk_bf16_f32) is the one rounding of the model.
__device__ __forceinline__ u32x4 hadamard8(const u32x4& a, const float* q) {
  u32x4 r;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t x = a[w];
    const bf16x2_t p = {(__bf16)(__uint_as_float(x << 16) * q[2 * w]),
                         (__bf16)(__uint_as_float(x & 0xffff0000u) * q[2 * w + 1])};
    r[w] = __builtin_bit_cast(uint32_t, p);
  }
  return r;
}


}  // namespace

// tokens per tile: 3 blocks of 32 (2304 tokens of a question make 24 tiles,
// so 16 questions x 24 tiles x 2 hidden tiles fill 256 CUs three times over)
constexpr int kMlpMT = 96;
constexpr int kMlpMB = kMlpMT / 32;   // 32-token blocks per tile
constexpr int kMlpKS = 32;       // columns of d per step (v part and v*q part)
constexpr int kMlpThreads = 512;
constexpr int kMlpPartial = 128; // hidden units per partial score (the narrowest tile)

// ---------------------------------------------------------------------------
// The per-question constant of the first layer.  Block (jt, qt): q_bar' of
// the questions qt*4 .. qt*4+3 is staged in LDS; wave w forms c_b[j] = sum_c W1[j][d + c] q_bar'_b[c] + b1[j]
// for its two hidden units j = 8*jt + 2*w + {0, 1} and the block's questions
// (products of two bf16 values are exact in float32; float32 sums).  The
// row loads of a 4096-column group are all issued before the products.
constexpr int kMlpPrepJ = 8;
constexpr int kMlpPrepQ = 4;
constexpr int kMlpMaxD = 8192;

__global__ void __launch_bounds__(256)
mlp_prep_kernel(const bf16_t* __restrict__ qbf, const bf16_t* __restrict__ W1,
                const float* __restrict__ b1, int B, int d, int h, float* __restrict__ cvec) {
  __shared__ __attribute__((aligned(16))) bf16_t qs[kMlpPrepQ][kMlpMaxD];
  const int jt = blockIdx.x, q0 = blockIdx.y * kMlpPrepQ;
  const int nq = min(kMlpPrepQ, B - q0);
  for (int i = threadIdx.x * 8; i < nq * d; i += blockDim.x * 8)
    *reinterpret_cast<u32x4*>(&qs[0][0] + (i / d) * kMlpMaxD + i % d) =
        *reinterpret_cast<const u32x4*>(qbf + (size_t)q0 * d + i);
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j0 = jt * kMlpPrepJ + wave * 2;
  const bf16_t* wr0 = W1 + (size_t)j0 * 3 * d + d;     // the q_bar block of row j0
  const bf16_t* wr1 = wr0 + (size_t)3 * d;
  float acc[2][kMlpPrepQ];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int qq = 0; qq < kMlpPrepQ; ++qq) acc[u][qq] = 0.f;
  for (int g = 0; g < d; g += 4096) {
    constexpr int CH = 4096 / 512;                     // 16-byte chunks per lane per group
    u32x4 w[2][CH];
#pragma unroll
    for (int t = 0; t < CH; ++t) {
      const int c = g + (t * 64 + lane) * 8;
      const bool ok = c < d;
      w[0][t] = ok ? *reinterpret_cast<const u32x4*>(wr0 + c) : u32x4{0u, 0u, 0u, 0u};
      w[1][t] = ok ? *reinterpret_cast<const u32x4*>(wr1 + c) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int t = 0; t < CH; ++t) {
      const int c = g + (t * 64 + lane) * 8;
      if (c >= d) continue;
      float w0[8], w1[8];
      unpack8_bf16(w[0][t], w0);
      unpack8_bf16(w[1][t], w1);
#pragma unroll
      for (int qq = 0; qq < kMlpPrepQ; ++qq) {
        if (qq >= nq) continue;
        float qv[8];
        unpack8_bf16(*reinterpret_cast<const u32x4*>(&qs[qq][c]), qv);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          acc[0][qq] = fmaf(w0[e], qv[e], acc[0][qq]);
          acc[1][qq] = fmaf(w1[e], qv[e], acc[1][qq]);
        }
      }
    }
  }
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int qq = 0; qq < kMlpPrepQ; ++qq) {
      const float v = wave_sum_f32(acc[u][qq]);
      if (lane == 0 && qq < nq)
        cvec[(size_t)(q0 + qq) * h + j0 + u] = v + (b1 ? b1[j0 + u] : 0.f);
    }
}

// ---------------------------------------------------------------------------
// W1's v block and Hadamard block, repacked in the order the score kernel's
// waves read them: for hidden tile nt (256 units), wave w (32 units), step s
// (32 columns), block x (0: v, 1: Hadamard), k16 sub-step kk and lane l, the
// 16 bytes W1[256 nt + 32 w + l % 32][x * 2d + 32 s + 8 (2 kk + l / 32) ...+7].
// One 1 KiB run per (nt, w, s, x, kk): every fragment load of the score kernel
// is one fully coalesced wave-wide load.
constexpr int kMlpNT = 256;

constexpr int kMlpPackBlocks = 1024;

__global__ void __launch_bounds__(256)
mlp_pack_kernel(const bf16_t* __restrict__ W1, int d, int h, u32x4* __restrict__ Wp,
                const double* __restrict__ qbar, bf16_t* __restrict__ qbf) {
  if ((int)blockIdx.x >= kMlpPackBlocks) {
    // q_bar' = bf16(float(q_bar)) of question blockIdx.x - kMlpPackBlocks
    const int b = blockIdx.x - kMlpPackBlocks;
    for (int c = threadIdx.x; c < d; c += blockDim.x)
      qbf[(size_t)b * d + c] = (bf16_t)f32_to_bf16((float)qbar[(size_t)b * d + c]);
    return;
  }
  const size_t total = (size_t)h * d / 4;            // 16-byte units of both blocks
  const int ksteps = d / kMlpKS;
  for (size_t u = (size_t)blockIdx.x * blockDim.x + threadIdx.x; u < total;
       u += (size_t)kMlpPackBlocks * blockDim.x) {
    const int l = (int)(u % 64);
    size_t r = u / 64;
    const int kk = (int)(r % 2); r /= 2;
    const int x = (int)(r % 2); r /= 2;
    const int s = (int)(r % ksteps); r /= ksteps;
    const int w = (int)(r % 8);
    const int nt = (int)(r / 8);
    const int j = nt * kMlpNT + w * 32 + (l & 31);
    const int col = x * 2 * d + s * kMlpKS + (2 * kk + (l >> 5)) * 8;
    Wp[u] = *reinterpret_cast<const u32x4*>(W1 + (size_t)j * 3 * d + col);
  }
}

// Work item = (question b, 96-token tile, 256-hidden tile); wave w of 8 owns
// hidden units 32 w .. 32 w + 31 of the tile for all 96 tokens (3 blocks of
// 32 x 32, v_mfma_f32_32x32x16_bf16).  Per 32-column step s:
//   * the v tile V[tile rows, 32 s : 32 s + 32] arrives in a 4-slot LDS ring
//     by direct global->LDS loads issued 3 steps ahead (16-byte chunks
//     XOR-swizzled by (row/2) % 4: operand reads of 8 consecutive rows hit
//     distinct banks);
//   * the workgroup forms the Hadamard tile bf16(v * q_bar') of step s+1 once,
//     into one of two LDS buffers, while it multiplies step s;
//   * each wave's W1 fragments come straight from the repacked weights into
//     registers, two steps ahead.
// The epilogue folds relu(a + c_b) . w2 and writes one partial of s_i per
// 128 hidden units.
constexpr int kMlpRing = 4;
constexpr int kMlpAhead = 3;

__global__ void __launch_bounds__(kMlpThreads)
mlp_score_kernel(const bf16_t* __restrict__ V, int N, int d, int B,
                 const u32x4* __restrict__ Wp, int h, const bf16_t* __restrict__ qbf,
                 const float* __restrict__ cvec, const float* __restrict__ w2,
                 float* __restrict__ sp, int n_items) {
  constexpr int A_ELEMS = kMlpMT * kMlpKS;       // 3072 (6 KiB)
  __shared__ __attribute__((aligned(1024))) bf16_t Ar[kMlpRing * A_ELEMS];
  __shared__ __attribute__((aligned(1024))) bf16_t Hd[2 * A_ELEMS];
  __shared__ __attribute__((aligned(16))) bf16_t Qs[kMlpMaxD];   // q_bar'_b

  const int per_xcd = gridDim.x / 8;
  const int item = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (item >= n_items) return;
  const int NTL = h / kMlpNT;
  const int MTL = (N + kMlpMT - 1) / kMlpMT;
  const int nt = item % NTL;
  const int mt = (item / NTL) % MTL;
  const int b = item / (NTL * MTL);
  const int i0 = mt * kMlpMT, j0 = nt * kMlpNT;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ksteps = d / kMlpKS;
  const int hh = lane >> 5, r32 = lane & 31;

  // the direct load of this thread's 16 bytes of a v tile: row tid/4,
  // physical chunk tid%4 holding logical chunk lc_t
  const int trow = tid >> 2;
  const int lc_t = (tid & 3) ^ ((trow >> 1) & 3);
  const bf16_t* vsrc = V + ((size_t)b * N + min(i0 + trow, N - 1)) * d + lc_t * 8;
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint32_t ar_lds = lds_addr(Ar) + (uint32_t)(wave_s * 1024);
  // (waves past the tile's rows, 4 * kMlpMT threads and up, copy nothing)
  const bool v_loader = tid < 4 * kMlpMT;
  auto issue_v = [&](int s) {
    if (v_loader)
      lds_dma16(vsrc + s * kMlpKS, __builtin_amdgcn_readfirstlane(
                                   ar_lds + (uint32_t)((s % kMlpRing) * A_ELEMS * 2)));
  };
  // Hadamard tile of step s (this thread's 8 values, same swizzled position;
  // q_bar' comes from LDS so that no vector-memory load joins the counted
  // queue of tile loads)
  auto hadamard_tile = [&](int s) {
    if (!v_loader) return;
    const u32x4 a = *reinterpret_cast<const u32x4*>(Ar + (s % kMlpRing) * A_ELEMS + tid * 8);
    float q[8];
    unpack8_bf16(*reinterpret_cast<const u32x4*>(Qs + s * kMlpKS + lc_t * 8), q);
    *reinterpret_cast<u32x4*>(Hd + (s & 1) * A_ELEMS + tid * 8) = hadamard8(a, q);
  };
  // W1 fragments of step s: [x][kk], x = 0 the v block, 1 the Hadamard block
  const u32x4* wsrc = Wp + ((size_t)(nt * 8 + wave) * ksteps) * 256 + lane;
  auto load_w = [&](int s, u32x4 (&w)[2][2]) {
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) w[x][kk] = wsrc[(size_t)s * 256 + (x * 2 + kk) * 64];
  };

  f32x16_t acc[kMlpMB];
#pragma unroll
  for (int mb = 0; mb < kMlpMB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[mb][v] = 0.f;

  // A operand offsets (elements) within a tile: block mb, k16 sub-step kk
  int aoff[2][kMlpMB];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int mb = 0; mb < kMlpMB; ++mb) {
      const int row = mb * 32 + r32;
      aoff[kk][mb] = row * kMlpKS + (((2 * kk + hh) ^ ((row >> 1) & 3)) << 3);
    }

  auto mma_step = [&](int s, const u32x4 (&w)[2][2]) {
    __builtin_amdgcn_sched_barrier(0);
    const bf16_t* At = Ar + (s % kMlpRing) * A_ELEMS;
    const bf16_t* Ht = Hd + (s & 1) * A_ELEMS;
    u32x4 a1[2][kMlpMB], a3[2][kMlpMB];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int mb = 0; mb < kMlpMB; ++mb) {
        a1[kk][mb] = *reinterpret_cast<const u32x4*>(At + aoff[kk][mb]);
        a3[kk][mb] = *reinterpret_cast<const u32x4*>(Ht + aoff[kk][mb]);
      }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int mb = 0; mb < kMlpMB; ++mb) {
        acc[mb] = mfma32_bf16(a1[kk][mb], w[0][kk], acc[mb]);
        acc[mb] = mfma32_bf16(a3[kk][mb], w[1][kk], acc[mb]);
      }
    // Schedule: half the operand reads ahead, then one MFMA per read, so the
    // read latency hides behind the matrix pipe.
    constexpr int NR = 4 * kMlpMB;             // operand reads (= MFMAs / 2)
    __builtin_amdgcn_sched_group_barrier(0x100, NR / 2, 0);
#pragma unroll
    for (int i = 0; i < NR / 2; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 3 * NR / 2, 0);
    __builtin_amdgcn_sched_barrier(0);
  };

  // prologue: q_bar'_b into LDS, v tiles of steps 0..2, W1 of steps 0 and 1,
  // Hadamard of step 0
  for (int c = tid * 8; c < d; c += kMlpThreads * 8)
    *reinterpret_cast<u32x4*>(Qs + c) =
        *reinterpret_cast<const u32x4*>(qbf + (size_t)b * d + c);
#pragma unroll
  for (int a = 0; a < kMlpAhead; ++a)
    if (a < ksteps) issue_v(a);
  u32x4 wA[2][2], wB[2][2];
  load_w(0, wA);
  load_w(min(1, ksteps - 1), wB);
  wait_vmcnt<0>();
  barrier_nofence();
  hadamard_tile(0);

  // Step s: wait for the v tile of step s+1 (the Hadamard pass reads it),
  // barrier (publishes it and the Hadamard tile of step s), load the v tile
  // of step s+3 into the slot step s-1 left, form the Hadamard tile of step
  // s+1, multiply step s, load the W1 fragments of step s+2.
  auto step = [&](int s, u32x4 (&w)[2][2]) {
    // outstanding per wave after this wait: the v tile of step s+2 (one
    // load, while there is one) and the W1 fragments of step s+1 (four loads)
    if (s + 2 < ksteps) wait_vmcnt<5>();
    else wait_vmcnt<4>();
    barrier_nofence();
    if (s + kMlpAhead < ksteps) issue_v(s + kMlpAhead);
    mma_step(s, w);
    if (s + 1 < ksteps) hadamard_tile(s + 1);
    // unconditional (the last steps reload the final step's fragments): a
    // conditional load would make the compiler drain the whole queue before
    // the next use of w
    load_w(min(s + 2, ksteps - 1), w);
  };
  int s = 0;
  for (; s + 1 < ksteps; s += 2) {
    step(s, wA);
    step(s + 1, wB);
  }
  if (s < ksteps) step(s, wA);

  // Epilogue: relu(a + c) * w2 for this lane's hidden unit, summed over the
  // 32 units of the wave, then over the four waves of each 128-unit part in
  // wave order.  Accumulator element v of block mb: token mb*32 + 8*(v/4) +
  // 4*hh + v%4; hidden unit j0 + 32*wave + r32.
  const int j = j0 + wave * 32 + r32;
  const float c = cvec[(size_t)b * h + j];
  const float wv = w2[j];
  float rs[kMlpMB][16];
#pragma unroll
  for (int mb = 0; mb < kMlpMB; ++mb)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float x = fmaxf(acc[mb][v] + c, 0.f) * wv;
#pragma unroll
      for (int o = 1; o < 32; o <<= 1) x += __shfl_xor(x, o, kWave);
      rs[mb][v] = x;
    }
  __syncthreads();                                   // the ring is free again
  float* red = reinterpret_cast<float*>(Ar);         // [8][128]
  if (r32 == 0) {
#pragma unroll
    for (int mb = 0; mb < kMlpMB; ++mb)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        red[wave * kMlpMT + mb * 32 + 8 * (v >> 2) + 4 * hh + (v & 3)] = rs[mb][v];
  }
  __syncthreads();
  if (tid < 2 * kMlpMT) {
    const int pp = tid / kMlpMT, row = tid % kMlpMT;
    if (i0 + row < N) {
      const float* rp = red + pp * 4 * kMlpMT + row;
      const float sum = ((rp[0] + rp[kMlpMT]) + rp[2 * kMlpMT]) + rp[3 * kMlpMT];
      sp[((size_t)(nt * 2 + pp) * B + b) * N + i0 + row] = sum;
    }
  }
}

// s_i = sum over hidden tiles of the partials (tile order) + b2.
__global__ void __launch_bounds__(256)
mlp_sum_kernel(const float* __restrict__ sp, int NTL, int B, int N, double b2,
               double* __restrict__ z, float* __restrict__ scores) {
  const int b = blockIdx.y;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= N) return;
  double s = 0.0;
  for (int t = 0; t < NTL; ++t) s += (double)sp[((size_t)t * B + b) * N + i];
  s += b2;
  z[(size_t)b * N + i] = s;
  if (scores) scores[(size_t)b * N + i] = (float)s;
}

static size_t mlp_align(size_t n) { return (n + 255) & ~(size_t)255; }

size_t mlp_scratch_bytes(const skip_problem_t& p, int hidden) {
  return mlp_align((size_t)p.B * p.d * sizeof(bf16_t)) +
         mlp_align((size_t)p.B * hidden * sizeof(float)) +
         mlp_align((size_t)(hidden / kMlpPartial) * p.B * (size_t)p.N * sizeof(float)) +
         mlp_align((size_t)hidden * 2 * p.d * sizeof(bf16_t));
}

MlpScratch carve_mlp_scratch(const skip_problem_t& p, int hidden, void* base) {
  char* c = static_cast<char*>(base);
  MlpScratch m;
  m.qbf = reinterpret_cast<bf16_t*>(c);
  c += mlp_align((size_t)p.B * p.d * sizeof(bf16_t));
  m.cvec = reinterpret_cast<float*>(c);
  c += mlp_align((size_t)p.B * hidden * sizeof(float));
  m.sp = reinterpret_cast<float*>(c);
  c += mlp_align((size_t)(hidden / kMlpPartial) * p.B * (size_t)p.N * sizeof(float));
  m.wpack = reinterpret_cast<u32x4*>(c);
  return m;
}

hipError_t launch_mlp_scores(const skip_problem_t& p, const skip_qvs_mlp_t& m, const void* V,
                             const double* qbar, MlpScratch ms, double* z, float* scores,
                             hipStream_t s) {
  const int h = m.hidden;
  // repacked weights and q_bar' (one launch), then the per-question constant
  hipLaunchKernelGGL(mlp_pack_kernel, dim3(kMlpPackBlocks + p.B), dim3(256), 0, s,
                     (const bf16_t*)m.W1, p.d, h, ms.wpack, qbar, ms.qbf);
  hipLaunchKernelGGL(mlp_prep_kernel, dim3(h / kMlpPrepJ, (p.B + kMlpPrepQ - 1) / kMlpPrepQ),
                     dim3(256), 0, s, (const bf16_t*)ms.qbf, (const bf16_t*)m.W1, m.b1, p.B,
                     p.d, h, ms.cvec);
  const int MTL = (p.N + kMlpMT - 1) / kMlpMT;
  const int n_items = p.B * MTL * (h / kMlpNT);
  const int grid = ((n_items + 7) / 8) * 8;
  hipLaunchKernelGGL(mlp_score_kernel, dim3(grid), dim3(kMlpThreads), 0, s, (const bf16_t*)V,
                     p.N, p.d, p.B, (const u32x4*)ms.wpack, h, (const bf16_t*)ms.qbf, ms.cvec,
                     m.w2, ms.sp, n_items);
  hipLaunchKernelGGL(mlp_sum_kernel, dim3((p.N + 255) / 256, p.B), dim3(256), 0, s, ms.sp,
                     h / kMlpPartial, p.B, p.N, m.b2, z, scores);
  return hipGetLastError();
}

}  // namespace skip

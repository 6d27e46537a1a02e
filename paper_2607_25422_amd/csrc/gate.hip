// Passage verification gate (paper App. B.4, Def. B.4; Alg. 1, verify step):
// for passage j of question b,
//   x_j = [q_bar ; v_bar ; e_j ; e_j * q_bar ; |e_j - q_bar|],
//   logit_j = w2 . relu(W x_j + b1) + b2,   nu_j = sigmoid(logit_j),
// and the question keeps, among its passages with nu_j >= tau, the
// ceil(rho * P_b) with the largest nu.  The model takes bf16 inputs (q_bar,
// v_bar, e_j rounded through float32; the product rounded from its exact
// value; the difference rounded from its float32 value).
//   gate_x_kernel      : the passage part of x_j, [e' ; (e' q')' ; |e' - q'|'],
//                        bf16, and the question part [q' ; v'] per question
//   gate_c_kernel      : c_b = W[:, 0:2d] [q'_b ; v'_b] + b1 (float32 sums of
//                        exact products)
//   gate_score_kernel  : W[:, 2d:5d] x_j on v_mfma_f32_32x32x16_bf16 for
//                        32 passages x 64 hidden units a workgroup (the four
//                        waves split the 3d columns), then relu(. + c_b) . w2
//                        summed over the 64 units: one partial logit per
//                        64-unit tile
//   gate_select_kernel : logit_j = sum of the partials + b2; threshold and
//                        top fraction per question (one wave a question)
#include <cmath>

#include "skip_common.h"
#include "skip_internal.h"

namespace skip {

namespace {

typedef __bf16 gbf16x8_t __attribute__((ext_vector_type(8)));
typedef float gf32x16_t __attribute__((ext_vector_type(16)));

__device__ __forceinline__ gf32x16_t gmfma(const u32x4& a, const u32x4& b, gf32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(gbf16x8_t, a),
                                                 __builtin_bit_cast(gbf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ void gunpack8(const u32x4& x, float* out) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    out[2 * w] = __uint_as_float(x[w] << 16);
    out[2 * w + 1] = __uint_as_float(x[w] & 0xffff0000u);
  }
}

// question of global passage index j (query_passages ascending)
__device__ __forceinline__ int question_of(const int32_t* qp, int B, int total, int j) {
  int lo = 0, hi = B;                      // answer in [0, B)
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (clampi(qp[mid], 0, total) <= j) lo = mid;
    else hi = mid;
  }
  return lo;
}

}  // namespace

constexpr int kGateMT = 32;       // passages per score tile
constexpr int kGateNT = 64;       // hidden units per score tile
constexpr int kGateCJ = 8;        // hidden units per c block (2 per wave)
constexpr int kGateCQ = 4;        // questions per c block (at most; LDS holds qpb x 2d bf16)

// Blocks [0, T): passage j = block: X[j] = [e' ; (e' q')' ; |e' - q'|'] and
// pq[j] = its question.  Blocks [T, T + B): QV[b] = [q'_b ; v'_b].
__global__ void __launch_bounds__(256)
gate_x_kernel(const double* __restrict__ qbar, const double* __restrict__ vbar,
              const double* __restrict__ kbar, const float* __restrict__ pkeys,
              const int32_t* __restrict__ query_passages, int B, int T, int d,
              bf16_t* __restrict__ X, bf16_t* __restrict__ QV, int32_t* __restrict__ pq) {
  const int blk = blockIdx.x;
  if (blk >= T) {
    const int b = blk - T;
    for (int c = threadIdx.x; c < d; c += blockDim.x) {
      QV[(size_t)b * 2 * d + c] = (bf16_t)f32_to_bf16((float)qbar[(size_t)b * d + c]);
      QV[(size_t)b * 2 * d + d + c] = (bf16_t)f32_to_bf16((float)vbar[(size_t)b * d + c]);
    }
    return;
  }
  const int j = blk;
  const int b = question_of(query_passages, B, T, j);
  if (threadIdx.x == 0) pq[j] = b;
  bf16_t* xr = X + (size_t)j * 3 * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    const float ev = pkeys ? pkeys[(size_t)j * d + c] : (float)kbar[(size_t)j * d + c];
    const float e = bf16_to_f32(f32_to_bf16(ev));
    const float q = bf16_to_f32(f32_to_bf16((float)qbar[(size_t)b * d + c]));
    xr[c] = (bf16_t)f32_to_bf16(e);
    xr[d + c] = (bf16_t)f32_to_bf16(e * q);            // exact product, one rounding
    xr[2 * d + c] = (bf16_t)f32_to_bf16(fabsf(e - q));  // float32 difference, one rounding
  }
}

// c_b[j] = W[j, 0:2d] . QV_b + b1[j] for hidden units j = 8*jt + 2*w + {0,1}
// and questions qpb*qt .. qpb*qt + qpb-1 (QV staged in LDS; float32 sums).
__global__ void __launch_bounds__(256)
gate_c_kernel(const bf16_t* __restrict__ QV, const bf16_t* __restrict__ W,
              const float* __restrict__ b1, int B, int d, int h, int qpb,
              float* __restrict__ cvec) {
  extern __shared__ __attribute__((aligned(16))) bf16_t qs[];   // [qpb][2d]
  const int jt = blockIdx.x, q0 = blockIdx.y * qpb;
  const int nq = min(qpb, B - q0);
  const int K = 2 * d;
  for (int i = threadIdx.x * 8; i < nq * K; i += blockDim.x * 8)
    *reinterpret_cast<u32x4*>(qs + i) = *reinterpret_cast<const u32x4*>(QV + (size_t)q0 * K + i);
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int j0 = jt * kGateCJ + wave * 2;
  const bf16_t* wr0 = W + (size_t)j0 * 5 * d;
  const bf16_t* wr1 = wr0 + (size_t)5 * d;
  float acc[2][kGateCQ];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int qq = 0; qq < kGateCQ; ++qq) acc[u][qq] = 0.f;
  for (int g = 0; g < K; g += 4096) {
    constexpr int CH = 4096 / 512;
    u32x4 w[2][CH];
#pragma unroll
    for (int t = 0; t < CH; ++t) {
      const int c = g + (t * 64 + lane) * 8;
      const bool ok = c < K;
      w[0][t] = ok ? *reinterpret_cast<const u32x4*>(wr0 + c) : u32x4{0u, 0u, 0u, 0u};
      w[1][t] = ok ? *reinterpret_cast<const u32x4*>(wr1 + c) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int t = 0; t < CH; ++t) {
      const int c = g + (t * 64 + lane) * 8;
      if (c >= K) continue;
      float w0[8], w1[8];
      gunpack8(w[0][t], w0);
      gunpack8(w[1][t], w1);
#pragma unroll
      for (int qq = 0; qq < kGateCQ; ++qq) {
        if (qq >= nq) continue;
        float qv[8];
        gunpack8(*reinterpret_cast<const u32x4*>(qs + qq * K + c), qv);
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
    for (int qq = 0; qq < kGateCQ; ++qq) {
      const float v = wave_sum_f32(acc[u][qq]);
      if (lane == 0 && qq < nq)
        cvec[(size_t)(q0 + qq) * h + j0 + u] = v + (b1 ? b1[j0 + u] : 0.f);
    }
}

// Tile (32 passages from 32*pt, 64 hidden units from 64*ht); the 3d passage
// columns are 3d/16 MFMA steps of 16 and wave w takes the steps w, w+4, ...
// Operands straight from global memory: A = X rows (lane: passage l%32, 8
// columns), B = W rows (lane: hidden unit l%32, 8 columns), four steps in
// flight per wave.
__global__ void __launch_bounds__(256)
gate_score_kernel(const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int T, int d,
                  int h, const int32_t* __restrict__ pq, const float* __restrict__ cvec,
                  const float* __restrict__ w2, float* __restrict__ part) {
  __shared__ float red[4][kGateMT][kGateNT + 1];
  const int pt = blockIdx.x, ht = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hh = lane >> 5, r32 = lane & 31;
  const int K = 3 * d;
  const int nsteps = K / 16;
  const int prow = min(pt * kGateMT + r32, T - 1);
  const bf16_t* xa = X + (size_t)prow * K + 8 * hh;
  const bf16_t* wb0 = W + (size_t)(ht * kGateNT + r32) * 5 * d + 2 * d + 8 * hh;
  const bf16_t* wb1 = wb0 + (size_t)32 * 5 * d;
  gf32x16_t acc[2];
#pragma unroll
  for (int v = 0; v < 16; ++v) { acc[0][v] = 0.f; acc[1][v] = 0.f; }
  constexpr int U = 4;
  int st = wave;
  for (; st + 4 * (U - 1) < nsteps; st += 4 * U) {
    u32x4 a[U], b0[U], b1[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = 16 * (st + 4 * u);
      a[u] = *reinterpret_cast<const u32x4*>(xa + k);
      b0[u] = *reinterpret_cast<const u32x4*>(wb0 + k);
      b1[u] = *reinterpret_cast<const u32x4*>(wb1 + k);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      acc[0] = gmfma(a[u], b0[u], acc[0]);
      acc[1] = gmfma(a[u], b1[u], acc[1]);
    }
  }
  for (; st < nsteps; st += 4) {
    const int k = 16 * st;
    const u32x4 a = *reinterpret_cast<const u32x4*>(xa + k);
    acc[0] = gmfma(a, *reinterpret_cast<const u32x4*>(wb0 + k), acc[0]);
    acc[1] = gmfma(a, *reinterpret_cast<const u32x4*>(wb1 + k), acc[1]);
  }
  // D layout: element v of block nb is passage 8*(v/4) + 4*hh + v%4, hidden
  // unit nb*32 + r32 of the tile
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int v = 0; v < 16; ++v)
      red[wave][8 * (v >> 2) + 4 * hh + (v & 3)][nb * 32 + r32] = acc[nb][v];
  __syncthreads();
  // thread t: passage t / 8, hidden units 8 * (t % 8) .. + 7
  const int m = threadIdx.x >> 3, n0 = (threadIdx.x & 7) * 8;
  const int p = pt * kGateMT + m;
  float s = 0.f;
  if (p < T) {
    const int b = pq[p];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int n = n0 + e, j = ht * kGateNT + n;
      const float a = ((red[0][m][n] + red[1][m][n]) + red[2][m][n]) + red[3][m][n];
      s += fmaxf(a + cvec[(size_t)b * h + j], 0.f) * w2[j];
    }
  }
  // sum over the 8 threads of a passage (consecutive lanes), fixed order
#pragma unroll
  for (int o = 1; o < 8; o <<= 1) s += __shfl_xor(s, o, kWave);
  if ((threadIdx.x & 7) == 0 && p < T) part[(size_t)ht * T + p] = s;
}

// One wave per question: logit_j = the float32 rounding of (the sum of the
// tile partials, in tile order, + b2); kept = verified (logit >= t) and among
// the cap largest verified logits (ties: lower index).  The cut is taken on
// the stored float32 logits, so it can be re-derived from them exactly.
__global__ void __launch_bounds__(64)
gate_select_kernel(const float* __restrict__ part, int NT, int T, int B,
                   const int32_t* __restrict__ query_passages, double b2, double t,
                   double rho, float* __restrict__ logits, uint8_t* __restrict__ keep) {
  __shared__ float z[64];
  __shared__ int ver[64];
  const int b = blockIdx.x, lane = threadIdx.x;
  int p0, p1;
  range_of(query_passages, b, T, p0, p1);
  const int P = min(p1 - p0, 64);
  float zl = 0.f;
  if (lane < P) {
    double acc = 0.0;
    for (int u = 0; u < NT; ++u) acc += (double)part[(size_t)u * T + p0 + lane];
    zl = (float)(acc + b2);
    if (logits) logits[p0 + lane] = zl;
  }
  z[lane] = zl;
  ver[lane] = (lane < P && (double)zl >= t) ? 1 : 0;
  __syncthreads();
  if (lane >= P) return;
  const int cap = (int)ceil(rho * (double)P - 1e-9);
  int rank = 0;
  for (int u = 0; u < P; ++u)
    if (ver[u] && (z[u] > zl || (z[u] == zl && u < lane))) ++rank;
  keep[p0 + lane] = (ver[lane] && rank < cap) ? 1u : 0u;
}

// v_bar of the fused route: the mean of V[b][kept_idx[r]] over the kept rows r
// of question b (0 when it has none).  Workgroup (512-column slice, question);
// wave w sums rows w, w+4, ... in float64, 16 bytes a lane; the four partial
// sums are combined in wave order through LDS.
__global__ void __launch_bounds__(256)
gate_vbar_kernel(const bf16_t* __restrict__ V, int N, int d, const int32_t* __restrict__ kept_offsets,
                 const int32_t* __restrict__ kept_idx, int total_kept,
                 double* __restrict__ vbar) {
  __shared__ double part[4][64][8];
  const int b = blockIdx.y, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = (blockIdx.x * 64 + lane) * 8;
  int r0, r1;
  range_of(kept_offsets, b, total_kept, r0, r1);
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  if (c < d) {
    const bf16_t* base = V + (size_t)b * N * d + c;
    for (int r = r0 + wave; r < r1; r += 4) {
      const int i = clampi(kept_idx[r], 0, N - 1);
      float x[8];
      gunpack8(*reinterpret_cast<const u32x4*>(base + (size_t)i * d), x);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += (double)x[e];
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[wave][lane][e] = acc[e];
  __syncthreads();
  if (wave != 0 || c >= d) return;
  const int L = r1 - r0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const double sum = ((part[0][lane][e] + part[1][lane][e]) + part[2][lane][e]) +
                       part[3][lane][e];
    vbar[(size_t)b * d + c + e] = L > 0 ? sum / (double)L : 0.0;
  }
}

hipError_t launch_gate_vbar(const skip_problem_t& p, const void* V,
                            const int32_t* kept_offsets, const int32_t* kept_idx,
                            GateScratch g, hipStream_t s) {
  hipLaunchKernelGGL(gate_vbar_kernel, dim3((p.d + 511) / 512, p.B), dim3(256), 0, s,
                     (const bf16_t*)V, p.N, p.d, kept_offsets, kept_idx, p.total_kept, g.vbar);
  return hipGetLastError();
}

static size_t galign(size_t n) { return (n + 255) & ~(size_t)255; }

size_t gate_scratch_bytes(const skip_problem_t& p, int hidden) {
  const size_t T = (size_t)p.total_passages;
  return galign((size_t)p.B * p.d * sizeof(double)) +        // vbar
         galign((size_t)p.B * p.d * sizeof(double)) +        // qbar
         galign(T * 3 * p.d * sizeof(bf16_t)) +               // X
         galign((size_t)p.B * 2 * p.d * sizeof(bf16_t)) +     // QV
         galign((size_t)p.B * hidden * sizeof(float)) +       // cvec
         galign((size_t)(hidden / kGateNT) * T * sizeof(float)) +   // partial logits
         galign(T * sizeof(int32_t));                         // question of each passage
}

GateScratch carve_gate_scratch(const skip_problem_t& p, int hidden, void* base) {
  const size_t T = (size_t)p.total_passages;
  char* c = static_cast<char*>(base);
  GateScratch g;
  g.vbar = reinterpret_cast<double*>(c);
  c += galign((size_t)p.B * p.d * sizeof(double));
  g.qbar = reinterpret_cast<double*>(c);
  c += galign((size_t)p.B * p.d * sizeof(double));
  g.X = reinterpret_cast<bf16_t*>(c);
  c += galign(T * 3 * p.d * sizeof(bf16_t));
  g.QV = reinterpret_cast<bf16_t*>(c);
  c += galign((size_t)p.B * 2 * p.d * sizeof(bf16_t));
  g.cvec = reinterpret_cast<float*>(c);
  c += galign((size_t)p.B * hidden * sizeof(float));
  g.part = reinterpret_cast<float*>(c);
  c += galign((size_t)(hidden / kGateNT) * T * sizeof(float));
  g.pq = reinterpret_cast<int32_t*>(c);
  return g;
}

hipError_t launch_gate(const skip_problem_t& p, const skip_skv_gate_t& gt, const double* qbar,
                       const double* kbar, const float* passage_keys,
                       const int32_t* query_passages, GateScratch g, float* logits,
                       uint8_t* keep, hipStream_t s) {
  const int T = p.total_passages, h = gt.hidden;
  if (T <= 0) return hipSuccess;
  hipLaunchKernelGGL(gate_x_kernel, dim3(T + p.B), dim3(256), 0, s, qbar, g.vbar, kbar,
                     passage_keys, query_passages, p.B, T, p.d, g.X, g.QV, g.pq);
  const int qpb = p.d <= 4096 ? kGateCQ : kGateCQ / 2;   // LDS at most 64 KiB
  const size_t lds = (size_t)qpb * 2 * p.d * sizeof(bf16_t);
  hipLaunchKernelGGL(gate_c_kernel, dim3(h / kGateCJ, (p.B + qpb - 1) / qpb), dim3(256), lds,
                     s, (const bf16_t*)g.QV, (const bf16_t*)gt.W, gt.b1, p.B, p.d, h, qpb,
                     g.cvec);
  hipLaunchKernelGGL(gate_score_kernel, dim3((T + kGateMT - 1) / kGateMT, h / kGateNT),
                     dim3(256), 0, s, (const bf16_t*)g.X, (const bf16_t*)gt.W, T, p.d, h,
                     (const int32_t*)g.pq, (const float*)g.cvec, gt.w2, g.part);
  const double t = std::log(gt.tau) - std::log1p(-gt.tau);
  hipLaunchKernelGGL(gate_select_kernel, dim3(p.B), dim3(64), 0, s, (const float*)g.part,
                     h / kGateNT, T, p.B, query_passages, gt.b2, t, gt.rho, logits, keep);
  return hipGetLastError();
}

}  // namespace skip

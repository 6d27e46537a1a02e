// Passage verification gate (paper App. B.4, Def. B.4; Alg. 1, verify step):
// for passage j of question b,
//   x_j = [q_bar ; v_bar ; e_j ; e_j * q_bar ; |e_j - q_bar|],
//   logit_j = w2 . relu(W x_j + b1) + b2,   nu_j = sigmoid(logit_j),
// and the question keeps, among its passages with nu_j >= tau, the
// ceil(rho * P_b) with the largest nu.  The model takes bf16 inputs (q_bar,
// v_bar, e_j rounded through float32; the product rounded from its exact
// value; the difference rounded from its float32 value).
//   gate_mean_kernel  : q_bar (question tokens) and v_bar (kept rows, given as
//                       rows or through kept_idx) in float64, 8 waves a
//                       workgroup, sixteen rows a wave in flight; then, per
//                       column slice, the bf16 gate inputs: the question
//                       blocks [q_bar ; v_bar] of every question, [B][2d],
//                       and the passage blocks [e ; e*q_bar ; |e - q_bar|]
//                       of every passage, [T][3d]
//   gate_score_kernel : W x on v_mfma_f32_32x32x16_bf16, split as
//                       W[:, 2d:5d] . (passage blocks) per passage plus
//                       W[:, 0:2d] . (question blocks) once per question (the
//                       same for all its passages); tiles of 64 rows x 64
//                       hidden units, the columns split into chunks (split-K,
//                       so the launch fills the chip at a few hundred
//                       passages); one float32 partial per chunk
//   gate_fin_kernel   : one workgroup a passage: its chunk partials in chunk
//                       order, then its question's in chunk order, + b1,
//                       relu, . w2, + b2 -> logit_j; the
//                       last workgroup of a question to finish (a counter in
//                       the workspace) takes the question's cut
#include <cmath>

#include "skip_common.h"
#include "skip_internal.h"

namespace skip {

constexpr int kGateRB = 2;         // 32-row MFMA blocks per score tile
constexpr int kGateMT = 32 * kGateRB;  // rows (passages or questions) per score tile
constexpr int kGateNT = 64;        // hidden units per score tile
constexpr int kGateMeanWaves = 8;  // waves per mean workgroup (256 columns)
constexpr int kGateTargetWG = 640; // passage-tile workgroups aimed for when choosing S
constexpr int kGateInFlight = 2;   // 64-column groups whose loads a wave issues together

// Workgroup (256-column slice, y): y < B is q_bar_y over the question tokens,
// y >= B is v_bar_{y-B} over the kept rows (rows[kept_offsets range], or
// V[b][kept_idx[r]] when kept_idx is given).  Row slot s of wave w is row
// w + 8s of the range; the half-wave s % 2 takes it, each lane 16 bytes of
// the row, so a half-wave covers the slice and a wave has two rows in each
// load instruction.  Sums in float64, sixteen slots (eight rows a half-wave)
// in flight; the sixteen partial sums are added in (wave, half) order; an
// empty range gives 0.
// The workgroup then writes its slice of the bf16 gate inputs: Xq[b] =
// [q' ; v'] (x' the bf16 rounding of float32(x)); a question workgroup also
// the slice of X[j] = [e' ; (e' q')' ; |e' - q'|'] for every passage j of
// its question (half-wave h taking the passages h, h+16, ...: the keys e_j
// are complete before this launch), pq[j] = b and, in slice 0, the
// question's finish counter cleared.
__global__ void __launch_bounds__(512)
gate_mean_kernel(const bf16_t* __restrict__ Qtok, const int32_t* __restrict__ q_offsets,
                 int total_qtok, const bf16_t* __restrict__ rows,
                 const int32_t* __restrict__ kept_offsets, const int32_t* __restrict__ kept_idx,
                 int N, int total_kept, int B, int d, double* __restrict__ qbar,
                 double* __restrict__ vbar, const double* __restrict__ kbar,
                 const float* __restrict__ pkeys, const int32_t* __restrict__ query_passages,
                 int T, bf16_t* __restrict__ X, bf16_t* __restrict__ Xq,
                 int32_t* __restrict__ pq, int32_t* __restrict__ done) {
  __shared__ double part[kGateMeanWaves][64][8];
  __shared__ float qsl[256];          // q' of the slice's columns (question workgroups)
  const bool isq = (int)blockIdx.y < B;
  const int b = isq ? (int)blockIdx.y : (int)blockIdx.y - B;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hf = lane >> 5, l32 = lane & 31;
  const int c = (blockIdx.x * 32 + l32) * 8;
  int r0, r1;
  if (isq) range_of(q_offsets, b, total_qtok, r0, r1);
  else range_of(kept_offsets, b, total_kept, r0, r1);
  const bf16_t* src = isq ? Qtok : rows;
  const bool indexed = !isq && kept_idx != nullptr;
  // indexed rows: lane i holds the index of the wave's i-th row (rows w,
  // w+8, ... up to 64 of them), read before the row loads that need it
  int my_idx = 0, base_r = r0 + wave;
  auto fetch_idx = [&](int rb) {
    const int r = rb + kGateMeanWaves * lane;
    my_idx = (indexed && r < r1) ? clampi(kept_idx[r], 0, N - 1) : 0;
    base_r = rb;
  };
  // every lane shuffles (the loop is wave-uniform); lanes past the last
  // column or the last row load nothing
  const bool cok = c < d;
  const u32x4 zero = {0u, 0u, 0u, 0u};
  auto load_row = [&](int r) -> u32x4 {
    size_t off = (size_t)r * d;
    if (indexed) {
      const int i = __shfl(my_idx, (r - base_r) / kGateMeanWaves, kWave);
      off = ((size_t)b * N + i) * d;
    }
    return (cok && r < r1)
               ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src + off + c))
               : zero;
  };
  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.0;
  constexpr int U = 16;                       // row slots a wave per round
  int r = r0 + wave;
  fetch_idx(r);
  for (; r < r1; r += kGateMeanWaves * U) {
    if (r + kGateMeanWaves * (U - 1) >= base_r + kGateMeanWaves * 64) fetch_idx(r);
    u32x4 x[U / 2];
#pragma unroll
    for (int u = 0; u < U / 2; ++u) x[u] = load_row(r + kGateMeanWaves * (2 * u + hf));
#pragma unroll
    for (int u = 0; u < U / 2; ++u) {
      if (r + kGateMeanWaves * (2 * u + hf) < r1) {
        float f[8];
        unpack8_bf16(x[u], f);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += (double)f[e];
      }
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[wave][lane][e] = acc[e];
  __syncthreads();
  const int L = r1 - r0;
  if (wave == 0 && hf == 0 && cok) {
    double* out = (isq ? qbar : vbar) + (size_t)b * d + c;
    float m[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      double s = part[0][l32][e] + part[0][l32 + 32][e];
#pragma unroll
      for (int w = 1; w < kGateMeanWaves; ++w) s = (s + part[w][l32][e]) + part[w][l32 + 32][e];
      const double mean = L > 0 ? s / (double)L : 0.0;
      out[e] = mean;
      m[e] = (float)mean;
    }
    u32x4 ob;
#pragma unroll
    for (int t = 0; t < 4; ++t) ob[t] = pack2_bf16(m[2 * t], m[2 * t + 1]);
    *reinterpret_cast<u32x4*>(Xq + (size_t)b * 2 * d + (isq ? 0 : d) + c) = ob;
    if (isq) {
#pragma unroll
      for (int e = 0; e < 8; ++e) qsl[8 * l32 + e] = bf16_to_f32(f32_to_bf16(m[e]));
    }
  }
  if (!isq) return;                   // uniform: the kind of workgroup
  if (blockIdx.x == 0 && threadIdx.x == 0) done[b] = 0;
  __syncthreads();
  int p0, p1;
  range_of(query_passages, b, T, p0, p1);
  for (int j = p0 + (int)(threadIdx.x >> 5); j < p1; j += 16) {
    if (blockIdx.x == 0 && l32 == 0) pq[j] = b;
    if (!cok) continue;
    float e[8];
    if (pkeys) {
      const float4 a = *reinterpret_cast<const float4*>(pkeys + (size_t)j * d + c);
      const float4 a2 = *reinterpret_cast<const float4*>(pkeys + (size_t)j * d + c + 4);
      e[0] = a.x; e[1] = a.y; e[2] = a.z; e[3] = a.w;
      e[4] = a2.x; e[5] = a2.y; e[6] = a2.z; e[7] = a2.w;
    } else {
      const double2* kp = reinterpret_cast<const double2*>(kbar + (size_t)j * d + c);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const double2 x = kp[t];
        e[2 * t] = (float)x.x;
        e[2 * t + 1] = (float)x.y;
      }
    }
    u32x4 oe, oh, od;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const float e0 = bf16_to_f32(f32_to_bf16(e[2 * t]));
      const float e1 = bf16_to_f32(f32_to_bf16(e[2 * t + 1]));
      const float q0 = qsl[8 * l32 + 2 * t], q1 = qsl[8 * l32 + 2 * t + 1];
      oe[t] = pack2_bf16(e0, e1);
      oh[t] = pack2_bf16(e0 * q0, e1 * q1);              // exact product, one rounding
      od[t] = pack2_bf16(fabsf(e0 - q0), fabsf(e1 - q1)); // float32 difference, one rounding
    }
    bf16_t* xr = X + (size_t)j * 3 * d;
    *reinterpret_cast<u32x4*>(xr + c) = oe;
    *reinterpret_cast<u32x4*>(xr + d + c) = oh;
    *reinterpret_cast<u32x4*>(xr + 2 * d + c) = od;
  }
}

// Row tiles: 64 passages (tiles 0 .. n_pt-1: the rows of X, K = 3d columns,
// against W's columns 2d .. 5d) or 64 questions (tiles n_pt ..: the rows of
// Xq, K = 2d, against W's columns 0 .. 2d), as two 32-row MFMA blocks that
// share every W operand.  Tile (rows, 64 hidden units), chunk z of its K
// columns, in groups of 64 columns: groups [z*ch, min((z+1)*ch, ceil(K/64))),
// wave w taking the groups w, w+4, ...; a question tile whose K ends before
// chunk z exits at once.  In a group the lane pair (row or unit l%32, half
// hh) reads the row's 128 contiguous bytes, 64 a lane as four 16-byte pieces,
// and piece u feeds MFMA step u: step u sums the columns 8u..8u+7 and
// 32+8u..32+8u+7 of the group (A and B take the same columns, so the product
// over the group is complete).  Two groups are in flight per wave, spare
// slots of the last round reading zeros.  A half group at the end of the
// columns (K/32 odd) reads zeros for its second half.  The four waves' sums are added in wave
// order and written as part[z][passage][unit] or partq[z][question][unit].
//
// Tiles go to XCDs by chunk: the hardware deals workgroup ids round-robin over
// the 8 XCDs, and id L takes chunk z = 8 * zl + L % 8 with (zl, ht, rt) the
// (L / 8)-th entry of that XCD's list, rt fastest.  Every tile of a chunk then
// runs on one XCD, whose L2 holds the chunk's columns of X and W, so each is
// read from memory once.  Ids whose chunk is past the last one exit at once.
__global__ void __launch_bounds__(256)
gate_score_kernel(const bf16_t* __restrict__ X, const bf16_t* __restrict__ Xq,
                  const bf16_t* __restrict__ W, int T, int B, int d, int h, int ch, int S,
                  float* __restrict__ part, float* __restrict__ partq) {
  __shared__ float red[4][kGateMT][kGateNT + 1];
  const int n_pt = (T + kGateMT - 1) / kGateMT, n_ht = h / kGateNT;
  const int n_rt = n_pt + (B + kGateMT - 1) / kGateMT;
  const int L = blockIdx.x, xcd = L & 7, jl = L >> 3;
  const int rt = jl % n_rt, ht = (jl / n_rt) % n_ht, zl = jl / (n_rt * n_ht);
  const int z = zl * 8 + xcd;
  if (z >= S) return;
  const bool qtile = rt >= n_pt;
  const int K = qtile ? 2 * d : 3 * d;
  const int ngroups = (K + 63) / 64;
  if (z * ch >= ngroups) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hh = lane >> 5, r32 = lane & 31;
  const int g1 = min((z + 1) * ch, ngroups);
  const int nrows = qtile ? B : T;
  const int r0 = (qtile ? rt - n_pt : rt) * kGateMT;
  const bf16_t* xbase = qtile ? Xq : X;
  const bf16_t* xa[kGateRB];
#pragma unroll
  for (int rb = 0; rb < kGateRB; ++rb)
    xa[rb] = xbase + (size_t)min(r0 + 32 * rb + r32, nrows - 1) * K + 32 * hh;
  const bf16_t* wb0 = W + (size_t)(ht * kGateNT + r32) * (5 * d) + (qtile ? 0 : 2 * d) + 32 * hh;
  const bf16_t* wb1 = wb0 + (size_t)32 * 5 * d;
  f32x16_t acc[kGateRB][2];
#pragma unroll
  for (int rb = 0; rb < kGateRB; ++rb)
#pragma unroll
    for (int v = 0; v < 16; ++v) { acc[rb][0][v] = 0.f; acc[rb][1][v] = 0.f; }
  const u32x4 zero = {0u, 0u, 0u, 0u};
  // group gg of the wave's rounds; past g1 (the last round's spare slots) zeros
  auto load_group = [&](int gg, u32x4 (*a)[4], u32x4* b0, u32x4* b1) {
    const int c = 64 * gg;
    const bool ok = gg < g1 && c + 32 * hh < K;   // K is a multiple of 32
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int rb = 0; rb < kGateRB; ++rb)
        a[rb][u] = ok ? *reinterpret_cast<const u32x4*>(xa[rb] + c + 8 * u) : zero;
      b0[u] = ok ? *reinterpret_cast<const u32x4*>(wb0 + c + 8 * u) : zero;
      b1[u] = ok ? *reinterpret_cast<const u32x4*>(wb1 + c + 8 * u) : zero;
    }
  };
  for (int g = z * ch + wave; g < g1; g += 4 * kGateInFlight) {
    u32x4 a[kGateInFlight][kGateRB][4], b0[kGateInFlight][4], b1[kGateInFlight][4];
#pragma unroll
    for (int e = 0; e < kGateInFlight; ++e) load_group(g + 4 * e, a[e], b0[e], b1[e]);
#pragma unroll
    for (int e = 0; e < kGateInFlight; ++e)
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int rb = 0; rb < kGateRB; ++rb) {
          acc[rb][0] = mfma32_bf16(a[e][rb][u], b0[e][u], acc[rb][0]);
          acc[rb][1] = mfma32_bf16(a[e][rb][u], b1[e][u], acc[rb][1]);
        }
  }
  // D layout: element v of block (rb, nb) is row 32*rb + 8*(v/4) + 4*hh + v%4,
  // hidden unit nb*32 + r32 of the tile
#pragma unroll
  for (int rb = 0; rb < kGateRB; ++rb)
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        red[wave][32 * rb + 8 * (v >> 2) + 4 * hh + (v & 3)][nb * 32 + r32] = acc[rb][nb][v];
  __syncthreads();
  // thread t: row t / (256 / MT), hidden units NPT * (t % (256 / MT)) .. + NPT-1
  constexpr int TPR = 256 / kGateMT, NPT = kGateNT / TPR;
  const int m = threadIdx.x / TPR, n0 = (threadIdx.x % TPR) * NPT;
  const int p = r0 + m;
  if (p >= nrows) return;
  float o[NPT];
#pragma unroll
  for (int e = 0; e < NPT; ++e) {
    const int n = n0 + e;
    o[e] = ((red[0][m][n] + red[1][m][n]) + red[2][m][n]) + red[3][m][n];
  }
  float4* dst = reinterpret_cast<float4*>((qtile ? partq : part) + ((size_t)z * nrows + p) * h +
                                          ht * kGateNT + n0);
#pragma unroll
  for (int e = 0; e < NPT / 4; ++e)
    dst[e] = make_float4(o[4 * e], o[4 * e + 1], o[4 * e + 2], o[4 * e + 3]);
}

// Block p (passage of question b, 512 threads): pre-activation of unit j =
// the S chunk partials of p in chunk order, then the Sq chunk partials of b
// in chunk order, + b1[j]; thread t sums relu(.) * w2[j] over its
// units j = t, t+512, ... in order; the eight waves' sums (wave shuffles, then
// wave order) plus b2, rounded to float32, are logit_p.  The block then bumps
// its question's counter; the block that completes it (P_b blocks in all)
// takes the cut: kept = logit >= t and among the cap largest verified logits
// (ties: lower index), on the float32 logits.
__global__ void __launch_bounds__(512)
gate_fin_kernel(const float* __restrict__ part, int S, const float* __restrict__ partq, int Sq,
                int T, int B, int h, const float* __restrict__ b1, const float* __restrict__ w2, double b2,
                const int32_t* __restrict__ pq, const int32_t* __restrict__ query_passages,
                double t, double rho, float* __restrict__ zbuf, int32_t* __restrict__ done,
                float* __restrict__ logits, uint8_t* __restrict__ keep) {
  __shared__ float wsum[8];
  __shared__ int last;
  const int p = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int b = pq[p];
  // a + src[0] + src[zs] + ... + src[(n-1) zs], in that order (loads issued
  // 16 at a time)
  auto chunk_sum = [](float a, const float* src, int n, size_t zs) {
    for (int zc = 0; zc < n; zc += 16) {
      float v[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] = zc + e < n ? src[(size_t)(zc + e) * zs] : 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (zc + e < n) a += v[e];
    }
    return a;
  };
  float s = 0.f;
  for (int j = threadIdx.x; j < h; j += blockDim.x) {
    float a = chunk_sum(0.f, part + (size_t)p * h + j, S, (size_t)T * h);
    a = chunk_sum(a, partq + (size_t)b * h + j, Sq, (size_t)B * h);
    a += b1 ? b1[j] : 0.f;
    s = fmaf(fmaxf(a, 0.f), w2[j], s);
  }
  s = wave_sum_f32(s);
  if (lane == 0) wsum[wave] = s;
  __syncthreads();
  int p0, p1;
  range_of(query_passages, b, T, p0, p1);
  const int P = min(p1 - p0, 64);
  if (threadIdx.x == 0) {
    double tot = (double)wsum[0];
    for (int w = 1; w < 8; ++w) tot += (double)wsum[w];
    tot += b2;
    const float zl = (float)tot;
    store_shared(&zbuf[p], zl);                   // read by the question's last block
    if (logits) logits[p] = zl;
  }
  // every block of the question done: the last one takes the cut
  if (!finish_and_check_last(&done[b], p1 - p0, &last) || wave != 0) return;
  // wave 0 of the question's last block: the cut with wave shuffles
  float zl = 0.f;
  if (lane < P) zl = load_shared(&zbuf[p0 + lane]);
  const int verified = (lane < P && (double)zl >= t) ? 1 : 0;
  const int cap = (int)ceil(rho * (double)P - 1e-9);
  int rank = 0;
  for (int u = 0; u < P; ++u) {
    const float zu = __shfl(zl, u, kWave);
    const int vu = __shfl(verified, u, kWave);
    if (vu && (zu > zl || (zu == zl && u < lane))) ++rank;
  }
  if (lane < P) keep[p0 + lane] = (verified && rank < cap) ? 1u : 0u;
}

static size_t galign(size_t n) { return (n + 255) & ~(size_t)255; }

// chunk length ch (64-column groups), chunk count S of the passage blocks'
// 3d columns and Sq of the question blocks' 2d columns (Sq <= S)
static void gate_split(int T, int h, int d, int* ch, int* S, int* Sq) {
  const int tiles = ((T + kGateMT - 1) / kGateMT) * (h / kGateNT);
  const int groups = (3 * d + 63) / 64;
  int s = (kGateTargetWG + tiles - 1) / tiles;
  const int smax = groups / 4 > 0 ? groups / 4 : 1;   // at least one group a wave
  s = s < 1 ? 1 : (s > smax ? smax : s);
  const int c = (groups + s - 1) / s;
  *ch = c;
  *S = (groups + c - 1) / c;
  *Sq = ((2 * d + 63) / 64 + c - 1) / c;
}

size_t gate_scratch_bytes(const skip_problem_t& p, int hidden) {
  const size_t T = (size_t)p.total_passages;
  int ch = 1, S = 1, Sq = 1;
  if (T > 0) gate_split((int)T, hidden, p.d, &ch, &S, &Sq);
  return 2 * galign((size_t)p.B * p.d * sizeof(double)) +          // qbar, vbar
         galign(T * 3 * p.d * sizeof(bf16_t)) +                     // X
         galign((size_t)p.B * 2 * p.d * sizeof(bf16_t)) +           // Xq
         galign((size_t)S * T * hidden * sizeof(float)) +           // passage chunk partials
         galign((size_t)Sq * p.B * hidden * sizeof(float)) +        // question chunk partials
         galign(T * sizeof(float)) +                                // logits
         galign(T * sizeof(int32_t)) +                              // question of each passage
         galign((size_t)p.B * sizeof(int32_t));                     // finish counters
}

GateScratch carve_gate_scratch(const skip_problem_t& p, int hidden, void* base) {
  const size_t T = (size_t)p.total_passages;
  int ch = 1, S = 1, Sq = 1;
  if (T > 0) gate_split((int)T, hidden, p.d, &ch, &S, &Sq);
  char* c = static_cast<char*>(base);
  GateScratch g;
  g.qbar = reinterpret_cast<double*>(c);
  c += galign((size_t)p.B * p.d * sizeof(double));
  g.vbar = reinterpret_cast<double*>(c);
  c += galign((size_t)p.B * p.d * sizeof(double));
  g.X = reinterpret_cast<bf16_t*>(c);
  c += galign(T * 3 * p.d * sizeof(bf16_t));
  g.Xq = reinterpret_cast<bf16_t*>(c);
  c += galign((size_t)p.B * 2 * p.d * sizeof(bf16_t));
  g.part = reinterpret_cast<float*>(c);
  c += galign((size_t)S * T * hidden * sizeof(float));
  g.partq = reinterpret_cast<float*>(c);
  c += galign((size_t)Sq * p.B * hidden * sizeof(float));
  g.z = reinterpret_cast<float*>(c);
  c += galign(T * sizeof(float));
  g.pq = reinterpret_cast<int32_t*>(c);
  c += galign(T * sizeof(int32_t));
  g.done = reinterpret_cast<int32_t*>(c);
  return g;
}

hipError_t launch_gate_means(const skip_problem_t& p, const void* Qtok,
                             const int32_t* q_offsets, const void* rows,
                             const int32_t* kept_offsets, const int32_t* kept_idx,
                             const double* kbar, const float* passage_keys,
                             const int32_t* query_passages, GateScratch g, hipStream_t s) {
  hipLaunchKernelGGL(gate_mean_kernel, dim3((p.d + 255) / 256, 2 * p.B), dim3(512), 0, s,
                     (const bf16_t*)Qtok, q_offsets, p.total_qtok, (const bf16_t*)rows,
                     kept_offsets, kept_idx, p.N, p.total_kept, p.B, p.d, g.qbar, g.vbar, kbar,
                     passage_keys, query_passages, p.total_passages, g.X, g.Xq, g.pq, g.done);
  return hipGetLastError();
}

hipError_t launch_gate(const skip_problem_t& p, const skip_skv_gate_t& gt,
                       const int32_t* query_passages, GateScratch g, float* logits,
                       uint8_t* keep, hipStream_t s) {
  const int T = p.total_passages, h = gt.hidden;
  if (T <= 0) return hipSuccess;
  int ch = 1, S = 1, Sq = 1;
  gate_split(T, h, p.d, &ch, &S, &Sq);
  const int n_rt = (T + kGateMT - 1) / kGateMT + (p.B + kGateMT - 1) / kGateMT;
  const int n_tiles = n_rt * (h / kGateNT);
  hipLaunchKernelGGL(gate_score_kernel, dim3(8 * ((S + 7) / 8) * n_tiles), dim3(256), 0, s,
                     (const bf16_t*)g.X, (const bf16_t*)g.Xq, (const bf16_t*)gt.W, T, p.B, p.d,
                     h, ch, S, g.part, g.partq);
  const double t = std::log(gt.tau) - std::log1p(-gt.tau);
  hipLaunchKernelGGL(gate_fin_kernel, dim3(T), dim3(512), 0, s, (const float*)g.part, S,
                     (const float*)g.partq, Sq, T, p.B, h, gt.b1, gt.w2, gt.b2,
                     (const int32_t*)g.pq, query_passages, t, gt.rho, g.z, g.done, logits, keep);
  return hipGetLastError();
}

}  // namespace skip

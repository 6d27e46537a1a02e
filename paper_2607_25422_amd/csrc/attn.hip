// Sparse cross-attention restricted to the bipartite graph (paper App. B.3,
// Def. B.3 attention rule; Alg. 1, fuse step).
//
// For kept row i of question b and head h, the logits run over every token of
// every passage adjacent to i (one 64-bit neighbour mask per row):
//   e_m = sm_scale * <Qh[i,h], Kh[m,h]>,  O = softmax(e) . Vh,  LSE = log sum exp e.
//
// bf16 path (MFMA).  Work item = (question b, head h, block of 128 kept rows):
// four waves, 32 rows each.  The item walks the passages adjacent to any of
// its rows, 64 tokens at a time.  K and V tiles of head h are staged once per
// item in LDS and shared by all 128 rows; the next tile is prefetched into
// registers while the current one is consumed.  Per wave:
//   S^T (64 tokens x 32 rows) = K_tile (64 x d_h) . Q^T   v_mfma_f32_32x32x16_bf16
//   rows not adjacent to the passage are masked to -inf (a wave with no
//   adjacent row skips the tile), online softmax in fp32 (base-2 exponent),
//   P rounded to bf16,
//   O^T (d_h x 32 rows) += V_tile^T . P^T                v_mfma_f32_32x32x16_bf16
// Computing the transposed products keeps each query row in one lane column,
// so row statistics need no cross-lane traffic except between the two half
// waves, and the S^T accumulator is already the P^T operand of the second
// product.  V is written to LDS transposed, with tokens permuted inside each
// 16-token block to match the S^T accumulator layout, so every MFMA operand
// is one 16-byte LDS read.
//
// Work items are laid out so that the row blocks of one (b, h) land on the
// same XCD (workgroups are dealt round-robin over the 8 XCDs), which keeps
// re-reads of a K/V tile within one L2.
//
// fp32 path: one wave per (kept row, head); 64 tokens per step, lane = token
// for the logits, lane = feature for the PV product.
#include "skip_common.h"
#include "skip_internal.h"

namespace skip {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kAttnRows = 128;   // kept rows per work item
constexpr int kTile = 64;        // tokens per K/V tile
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16_t mfma32(const u32x4& a, const u32x4& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  return f32_to_bf16(lo) | (f32_to_bf16(hi) << 16);
}

// Position of token w (0..63) of a tile inside its 16-token block of the
// transposed V tile: the S^T accumulator gives lane half hh, element e the
// token 8*(e/4) + 4*hh + e%4 of the block, and that pair is stored at 8*hh + e.
__device__ __forceinline__ int vt_pos(int w) {
  const int blk = w >> 4, ww = w & 15;
  const int hh = (ww >> 2) & 1;
  const int e = 4 * (ww >> 3) + (ww & 3);
  return 16 * blk + 8 * hh + e;
}

template <int D>
__global__ void __launch_bounds__(256)
attn_bf16_kernel(const bf16_t* __restrict__ qbase, const int32_t* __restrict__ kept_idx,
                 int N, int qstride, const int32_t* __restrict__ kept_offsets,
                 const bf16_t* __restrict__ Kh, const bf16_t* __restrict__ Vh,
                 const int32_t* __restrict__ passage_offsets,
                 const int32_t* __restrict__ query_passages,
                 const uint64_t* __restrict__ rowmask, int H, int total_kept,
                 int total_passages, int total_tokens, int k_max, int P_max, int RB,
                 int n_items, float scale_log2, void* __restrict__ O, int o_f32,
                 float* __restrict__ lse) {
  constexpr int KS = D + 8;              // K tile row stride (elements)
  constexpr int VS = kTile + 8;          // V^T tile row stride (elements)
  constexpr int KB = D / 16;             // k-blocks of the QK^T product
  constexpr int DT = D / 32;             // 32-wide feature tiles of O
  constexpr int CH = kTile * D / 8;      // 16-byte chunks per tile
  constexpr int CPT = CH / 256;          // chunks per thread
  static_assert(CH % 256 == 0, "tile chunks must divide over the workgroup");
  __shared__ __attribute__((aligned(16))) bf16_t Ks[kTile * KS];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[D * VS];
  __shared__ uint64_t wave_union[4];

  // XCD-aware decode: consecutive items on one XCD share (b, h).
  const int per_xcd = gridDim.x / 8;
  const int item = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (item >= n_items) return;
  const int rb = item % RB;
  const int h = (item / RB) % H;
  const int b = item / (RB * H);

  int k0, k1, p0, p1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  range_of(query_passages, b, total_passages, p0, p1);
  const int kq = min(k1 - k0, k_max);
  const int P = min(min(p1 - p0, P_max), 64);
  const int row0 = rb * kAttnRows;
  if (row0 >= kq) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int col = lane & 31;         // query row within the wave
  const int hh = lane >> 5;          // half wave
  const int r = row0 + wave * 32 + col;
  const bool row_ok = r < kq;

  uint64_t mrow = row_ok ? rowmask[k0 + r] : 0ull;
  if (P < 64) mrow &= (1ull << P) - 1ull;
  uint64_t wmask = mrow;
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) wmask |= __shfl_xor(wmask, s, 64);
  if (lane == 0) wave_union[wave] = wmask;

  // Q^T fragments (B operand): row `col`, features kb*16 + 8*hh .. +7.
  u32x4 qf[KB];
  {
    const bf16_t* qrow = nullptr;
    if (row_ok) {
      if (kept_idx) {
        const int src = clampi(kept_idx[k0 + r], 0, N - 1);
        qrow = qbase + ((size_t)b * N + src) * qstride + (size_t)h * D;
      } else {
        qrow = qbase + (size_t)(k0 + r) * qstride + (size_t)h * D;
      }
    }
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
      qf[kb] = row_ok ? *reinterpret_cast<const u32x4*>(qrow + kb * 16 + 8 * hh)
                      : u32x4{0u, 0u, 0u, 0u};
  }
  __syncthreads();
  const uint64_t U = wave_union[0] | wave_union[1] | wave_union[2] | wave_union[3];

  f32x16_t acc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[t][v] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  // Tile walk over (adjacent passage, 64-token block).
  uint64_t urem = U;
  int cur_j = -1, cur_t = 0, cur_end = 0;
  auto advance = [&]() -> bool {
    if (cur_j >= 0 && cur_t + kTile < cur_end) {
      cur_t += kTile;
      return true;
    }
    while (urem) {
      const int j = __builtin_ctzll(urem);
      urem &= urem - 1ull;
      int ts, te;
      range_of(passage_offsets, p0 + j, total_tokens, ts, te);
      if (te > ts) {
        cur_j = j; cur_t = ts; cur_end = te;
        return true;
      }
    }
    return false;
  };

  u32x4 kreg[CPT], vreg[CPT];
  auto load_tile = [&](int t_base, int t_end) {
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int ch = tid + 256 * c;
      const int tok = ch / (D / 8), c8 = ch % (D / 8);
      const int t = t_base + tok;
      if (t < t_end) {
        const size_t off = ((size_t)t * H + h) * D + c8 * 8;
        kreg[c] = *reinterpret_cast<const u32x4*>(Kh + off);
        vreg[c] = *reinterpret_cast<const u32x4*>(Vh + off);
      } else {
        kreg[c] = u32x4{0u, 0u, 0u, 0u};
        vreg[c] = u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      const int ch = tid + 256 * c;
      const int tok = ch / (D / 8), c8 = ch % (D / 8);
      *reinterpret_cast<u32x4*>(&Ks[tok * KS + c8 * 8]) = kreg[c];
      const int pos = vt_pos(tok);
      const uint32_t w4[4] = {vreg[c].x, vreg[c].y, vreg[c].z, vreg[c].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        Vt[(c8 * 8 + 2 * e) * VS + pos] = (bf16_t)(w4[e] & 0xffffu);
        Vt[(c8 * 8 + 2 * e + 1) * VS + pos] = (bf16_t)(w4[e] >> 16);
      }
    }
  };

  bool have = advance();
  if (have) load_tile(cur_t, cur_end);
  while (have) {
    const int j = cur_j, t_base = cur_t, t_end = cur_end;
    __syncthreads();
    store_tile();
    __syncthreads();
    have = advance();
    if (have) load_tile(cur_t, cur_end);

    if ((wmask >> j) & 1ull) {
      const bool adj = (mrow >> j) & 1ull;
      f32x16_t s[2];
#pragma unroll
      for (int st = 0; st < 2; ++st) {
#pragma unroll
        for (int v = 0; v < 16; ++v) s[st][v] = 0.f;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
          const u32x4 a =
              *reinterpret_cast<const u32x4*>(&Ks[(st * 32 + col) * KS + kb * 16 + 8 * hh]);
          s[st] = mfma32(a, qf[kb], s[st]);
        }
      }
      // mask + scale, tile max
      float mt = -INFINITY;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int tok = t_base + st * 32 + 8 * (v >> 2) + 4 * hh + (v & 3);
          const float x = (adj && tok < t_end) ? s[st][v] * scale_log2 : -INFINITY;
          s[st][v] = x;
          mt = fmaxf(mt, x);
        }
      mt = fmaxf(mt, __shfl_xor(mt, 32, 64));
      const float m_new = fmaxf(m_run, mt);
      const float alpha = (m_new == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
      float ls = 0.f;
      u32x4 pb[4];
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        float pv[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float x = s[st][v];
          pv[v] = (x == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(x - m_new);
          ls += pv[v];
        }
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          pb[2 * st + g] = u32x4{pack2_bf16(pv[8 * g + 0], pv[8 * g + 1]),
                                 pack2_bf16(pv[8 * g + 2], pv[8 * g + 3]),
                                 pack2_bf16(pv[8 * g + 4], pv[8 * g + 5]),
                                 pack2_bf16(pv[8 * g + 6], pv[8 * g + 7])};
        }
      }
      l_run = l_run * alpha + ls;
      m_run = m_new;
#pragma unroll
      for (int t = 0; t < DT; ++t) {
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[t][v] *= alpha;
#pragma unroll
        for (int kb2 = 0; kb2 < 4; ++kb2) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(
              &Vt[(t * 32 + col) * VS + 16 * kb2 + 8 * hh]);
          acc[t] = mfma32(a, pb[kb2], acc[t]);
        }
      }
    }
  }

  // finalize
  const float l_tot = l_run + __shfl_xor(l_run, 32, 64);
  if (!row_ok) return;
  const float inv = (l_tot > 0.f) ? 1.f / l_tot : 0.f;
  const size_t obase = ((size_t)(k0 + r) * H + h) * D;
  if (o_f32) {
    float* orow = static_cast<float*>(O) + obase;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int f = t * 32 + 8 * g + 4 * hh;
        float4 w = make_float4(acc[t][4 * g + 0] * inv, acc[t][4 * g + 1] * inv,
                               acc[t][4 * g + 2] * inv, acc[t][4 * g + 3] * inv);
        *reinterpret_cast<float4*>(orow + f) = w;
      }
  } else {
    bf16_t* orow = static_cast<bf16_t*>(O) + obase;
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int f = t * 32 + 8 * g + 4 * hh;
        uint2 w;
        w.x = pack2_bf16(acc[t][4 * g + 0] * inv, acc[t][4 * g + 1] * inv);
        w.y = pack2_bf16(acc[t][4 * g + 2] * inv, acc[t][4 * g + 3] * inv);
        *reinterpret_cast<uint2*>(orow + f) = w;
      }
  }
  if (lse && hh == 0)
    lse[(size_t)(k0 + r) * H + h] = (l_tot > 0.f) ? (m_run + log2f(l_tot)) * kLn2 : -INFINITY;
}

// ---------------------------------------------------------------------------
// fp32 path: one wave per (kept row, head).
template <int D>
__global__ void __launch_bounds__(256)
attn_f32_kernel(const float* __restrict__ qbase, const int32_t* __restrict__ kept_idx, int N,
                int qstride, const int32_t* __restrict__ kept_offsets,
                const float* __restrict__ Kh, const float* __restrict__ Vh,
                const int32_t* __restrict__ passage_offsets,
                const int32_t* __restrict__ query_passages,
                const uint64_t* __restrict__ rowmask, int H, int total_kept,
                int total_passages, int total_tokens, int k_max, int P_max, float sm_scale,
                float* __restrict__ O, float* __restrict__ lse) {
  constexpr int E = D / 64;            // features per lane
  __shared__ float qs[4][D];
  __shared__ float ps[4][64];
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int k0, k1, p0, p1;
  range_of(kept_offsets, b, total_kept, k0, k1);
  range_of(query_passages, b, total_passages, p0, p1);
  const int kq = min(k1 - k0, k_max);
  const int P = min(min(p1 - p0, P_max), 64);
  const int item = blockIdx.x * 4 + wave;
  const int r = item / H, h = item % H;
  if (r >= kq) return;                  // whole wave; no block barrier below

  const float* qrow;
  if (kept_idx) {
    const int src = clampi(kept_idx[k0 + r], 0, N - 1);
    qrow = qbase + ((size_t)b * N + src) * qstride + (size_t)h * D;
  } else {
    qrow = qbase + (size_t)(k0 + r) * qstride + (size_t)h * D;
  }
#pragma unroll
  for (int e = 0; e < E; ++e) qs[wave][lane * E + e] = qrow[lane * E + e];
  __builtin_amdgcn_wave_barrier();

  uint64_t m = rowmask[k0 + r];
  if (P < 64) m &= (1ull << P) - 1ull;
  float m_run = -INFINITY, l_run = 0.f;
  float o[E];
#pragma unroll
  for (int e = 0; e < E; ++e) o[e] = 0.f;
  while (m) {
    const int j = __builtin_ctzll(m);
    m &= m - 1ull;
    int ts, te;
    range_of(passage_offsets, p0 + j, total_tokens, ts, te);
    for (int t0 = ts; t0 < te; t0 += 64) {
      const int t = t0 + lane;
      float x = -INFINITY;
      if (t < te) {
        const float* krow = Kh + ((size_t)t * H + h) * D;
        float s = 0.f;
        for (int c = 0; c < D; ++c) s = fmaf(qs[wave][c], krow[c], s);
        x = s * sm_scale;
      }
      const float m_new = fmaxf(m_run, wave_max_f32(x));
      const float alpha = (m_run == -INFINITY) ? 0.f : expf(m_run - m_new);
      const float p = (x == -INFINITY) ? 0.f : expf(x - m_new);
      l_run = l_run * alpha + wave_sum_f32(p);
      m_run = m_new;
      ps[wave][lane] = p;
      __builtin_amdgcn_wave_barrier();
      const int n = min(64, te - t0);
#pragma unroll
      for (int e = 0; e < E; ++e) {
        float a = o[e] * alpha;
        for (int q = 0; q < n; ++q)
          a = fmaf(ps[wave][q], Vh[((size_t)(t0 + q) * H + h) * D + lane * E + e], a);
        o[e] = a;
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  const float inv = (l_run > 0.f) ? 1.f / l_run : 0.f;
  float* orow = O + ((size_t)(k0 + r) * H + h) * D;
#pragma unroll
  for (int e = 0; e < E; ++e) orow[lane * E + e] = o[e] * inv;
  if (lse && lane == 0)
    lse[(size_t)(k0 + r) * H + h] = (l_run > 0.f) ? m_run + logf(l_run) : -INFINITY;
}

// ---------------------------------------------------------------------------
hipError_t launch_attention(const skip_problem_t& p, QuerySource q,
                            const int32_t* kept_offsets, const void* Kh, const void* Vh,
                            const int32_t* passage_offsets, const int32_t* query_passages,
                            const uint64_t* rowmask, void* O, float* lse, hipStream_t s) {
  if (p.k_max <= 0) return hipSuccess;
  const int qstride = p.d;
  if (p.dtype == SKIP_BF16) {
    const int RB = (p.k_max + kAttnRows - 1) / kAttnRows;
    const int n_items = p.B * p.H * RB;
    const int grid = ((n_items + 7) / 8) * 8;
    const float sl2 = p.sm_scale * kLog2e;
#define SKIP_ATTN_BF16(DD)                                                                   \
  hipLaunchKernelGGL(attn_bf16_kernel<DD>, dim3(grid), dim3(256), 0, s,                      \
                     (const bf16_t*)q.base, q.kept_idx, q.N, qstride, kept_offsets,          \
                     (const bf16_t*)Kh, (const bf16_t*)Vh, passage_offsets, query_passages,  \
                     rowmask, p.H, p.total_kept, p.total_passages, p.total_tokens, p.k_max,  \
                     p.P_max, RB, n_items, sl2, O, p.o_f32, lse)
    if (p.d_h == 64) SKIP_ATTN_BF16(64);
    else SKIP_ATTN_BF16(128);
#undef SKIP_ATTN_BF16
  } else {
    dim3 grid((p.k_max * p.H + 3) / 4, p.B);
#define SKIP_ATTN_F32(DD)                                                                    \
  hipLaunchKernelGGL(attn_f32_kernel<DD>, grid, dim3(256), 0, s, (const float*)q.base,       \
                     q.kept_idx, q.N, qstride, kept_offsets, (const float*)Kh,               \
                     (const float*)Vh, passage_offsets, query_passages, rowmask, p.H,        \
                     p.total_kept, p.total_passages, p.total_tokens, p.k_max, p.P_max,       \
                     p.sm_scale, (float*)O, lse)
    if (p.d_h == 64) SKIP_ATTN_F32(64);
    else SKIP_ATTN_F32(128);
#undef SKIP_ATTN_F32
  }
  return hipGetLastError();
}

}  // namespace skip

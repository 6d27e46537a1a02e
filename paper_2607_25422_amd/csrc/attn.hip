// Sparse cross-attention restricted to the bipartite graph (paper App. B.3,
// Def. B.3 attention rule; Alg. 1, fuse step).
//
// For kept row i of question b and head h, the logits run over every token of
// every passage adjacent to i (one 64-bit neighbour mask per row):
//   e_m = sm_scale * <Qh[i,h], Kh[m,h]>,  O = softmax(e) . Vh,  LSE = log sum exp e.
//
// bf16 path (MFMA).  Work item = (question b, head h, block of <= 256 kept
// rows), eight waves.  The item walks the passages adjacent to any of its
// rows, 64 tokens at a time; K and V tiles of head h are staged once per item
// in an LDS ring and shared by all rows.  Per wave and tile:
//   S^T (tokens x 32 rows) = K_tile (tokens x d_h) . Q^T   v_mfma_f32_32x32x16_bf16
//   rows not adjacent to the passage are masked to -inf, online softmax in
//   fp32 (base-2 exponent), P rounded to bf16,
//   O^T (d_h x 32 rows) += V_tile^T . P^T                  v_mfma_f32_32x32x16_bf16
// Computing the transposed products keeps each query row in one lane column,
// so row statistics need no cross-lane traffic except between the two half
// waves, and the S^T accumulator is already the P^T operand of the second
// product.  The V^T operand comes from transposing LDS reads in the token
// order of the S^T accumulator layout.
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
typedef short s16x4_t __attribute__((ext_vector_type(4)));
template <int N>
struct IntC {                     // a compile-time count passed to a generic lambda
  static constexpr int value = N;
};

constexpr int kWaves = 8;                 // waves per work item
constexpr int kThreads = 64 * kWaves;
constexpr int kMaxRows = 32 * kWaves;     // kept rows per work item
constexpr int kTile = 64;                 // tokens per K/V tile
constexpr int kStages = 4;                // K/V tiles resident in LDS
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16_t mfma32(const u32x4& a, const u32x4& b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two floats -> packed bf16 pair, round-to-nearest-even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack2_bf16(float lo, float hi) {
  bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

// Wait until at most N of this wave's vector-memory operations are pending
// (expcnt and lgkmcnt left unconstrained).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Workgroup barrier without a memory fence: LDS in the loop is written only
// by direct global->LDS loads, whose completion is awaited explicitly.
__device__ __forceinline__ void barrier_nofence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// LDS byte address of a shared-memory pointer, as a wave-uniform value.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p);
}

// A wave-uniform 64-bit value moved to scalar registers.
__device__ __forceinline__ uint64_t uniform64(uint64_t x) {
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Direct global->LDS load of 16 bytes per lane (global_load_lds_dwordx4):
// lane l's bytes land at LDS byte address lds + 16 * l (lds wave-uniform).
// Issued through inline assembly so that the compiler's wait-count pass does
// not treat it as a write that may alias every later LDS read (it would put
// a full vmcnt(0) before them and drain the prefetch ring); completion is
// awaited explicitly with wait_vmem<> before the barrier that publishes a
// tile.
__device__ __forceinline__ void lds_dma16(const void* g, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(g), "s"(lds)
               : "memory", "m0");
}

// Value of lane l ^ 32 (v_permlane32_swap: the two half-waves trade places).
__device__ __forceinline__ float swap_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                  false, false);
  return __uint_as_float(__lane_id() < 32 ? r[1] : r[0]);
}

// Transposing LDS read: in each group of 16 lanes, lane j receives element
// j & 3 of the 8-byte pieces addressed by lanes (j >> 2) + 4e, e = 0..3.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ u32x2 ds_read_tr16(const bf16_t* p) {
  s16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4_t*)(p));
  return __builtin_bit_cast(u32x2, v);
}

// bf16 path.  Work item = (question b, head h, block of <= 256 kept rows);
// eight waves, 32 rows each.  K and V tiles of 64 tokens of head h stream
// through a 4-stage LDS ring filled by direct global->LDS loads (16 bytes a
// lane), three tiles ahead of the tile being consumed, one barrier per tile.
// Tiles are stored in natural token-major layout with 16-byte chunks XOR-
// swizzled by row (conflict-free MFMA operand reads).  Per wave and tile:
//   S^T (64 tokens x 32 rows) = K_tile . Q^T     (A: K rows, 16-byte LDS reads)
//   mask rows without an edge to the passage and tokens past its end, online
//   softmax in fp32 (base-2), P rounded to bf16,
//   O^T (d_h x 32 rows) += V_tile^T . P^T        (A: V^T via transposing LDS reads)
// The S^T accumulator layout gives lane half hh, element e of a 16-token
// block the token 8*(e/4) + 4*hh + e%4; the V^T operand is read in that same
// token order, so P^T needs no data movement.
template <int D, bool SPLIT_P>
__global__ void __launch_bounds__(kThreads)
attn_bf16_kernel(const bf16_t* __restrict__ qbase, const int32_t* __restrict__ kept_idx,
                 int N, int qstride, const int32_t* __restrict__ kept_offsets,
                 const bf16_t* __restrict__ Kh, const bf16_t* __restrict__ Vh,
                 const int32_t* __restrict__ passage_offsets,
                 const int32_t* __restrict__ query_passages,
                 const uint64_t* __restrict__ rowmask, int H, int total_kept,
                 int total_passages, int total_tokens, int k_max, int P_max, int RB,
                 int n_items, float scale_log2, void* __restrict__ O, int o_f32,
                 float* __restrict__ lse) {
  constexpr int NCH = D / 8;               // 16-byte chunks per token row
  constexpr int KB = D / 16;               // k-blocks of QK^T
  constexpr int DT = D / 32;               // 32-wide feature tiles of O
  constexpr int TILE = kTile * D;          // elements per K (or V) tile
  constexpr int NI = kTile * NCH / 64;     // 1 KiB load instructions per K (or V) tile
  // direct loads per lane per tile (waves >= NI issue none when NI < kWaves)
  constexpr int kLoaders = kWaves / 2;    // group A issues every tile load
  constexpr int LPT = 2 * ((NI + kLoaders - 1) / kLoaders);
  // V chunk swizzle: depends on row % 4 only; keeps the transposing reads of
  // four consecutive tokens on distinct banks.
  auto vswz = [](int row) { return (NCH >= 16 ? 4 : 2) * (row & 3); };
  static_assert(NI % kLoaders == 0, "tile loads must divide over the loading waves");
  static_assert(2 * (DT * 16 + 2) * 64 * 4 <= kStages * TILE * 2,
                "the merge of split blocks reuses the K ring");
  __shared__ __attribute__((aligned(1024))) bf16_t Kbuf[kStages * TILE];
  __shared__ __attribute__((aligned(1024))) bf16_t Vbuf[kStages * TILE];
  __shared__ uint64_t wave_union[kWaves];
  __shared__ int p_ts[64], p_te[64];

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
  const int nblk = (kq + kMaxRows - 1) / kMaxRows;
  if (rb >= nblk) return;
  const int rpb = ((kq + nblk - 1) / nblk + 31) / 32 * 32;   // rows per block
  const int row0 = rb * rpb;
  const int row_end = min(kq, row0 + rpb);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int col = lane & 31;         // query row within the wave
  const int hh = lane >> 5;          // half wave
  // Waves w and w+4 share a SIMD.  A wave takes one 32-row block over whole
  // tiles, or one 32-token half of every tile of a block (its partner, wave
  // w^1, takes the other half; the two merge once at the end).  Halves are
  // used where they even out the rows per SIMD: 5-6 blocks (waves 4-7 split
  // blocks 4 and 5: 48 rows per SIMD instead of 64) and 1-2 blocks (one
  // block over two SIMDs).
  const int nrb = (row_end - row0 + 31) / 32;
  int wb = wave, half = -1;          // wave's row block; half < 0: whole tiles
  if (nrb <= 2) {
    wb = wave >> 1;
    half = wave & 1;
  } else if ((nrb == 5 || nrb == 6) && wave >= 4) {
    wb = 4 + ((wave - 4) >> 1);
    half = wave & 1;
  }
  const bool any_split = nrb <= 2 || nrb == 5 || nrb == 6;   // uniform over the item
  const bool split = half >= 0;
  const int sub0 = split ? half : 0;                           // first 32-token sub-tile
  const int r = row0 + wb * 32 + col;
  const bool row_ok = wb < nrb && r < row_end;

  if (tid < P) {
    int ts, te;
    range_of(passage_offsets, p0 + tid, total_tokens, ts, te);
    p_ts[tid] = ts;
    p_te[tid] = te;
  }
  uint64_t mrow = row_ok ? rowmask[k0 + r] : 0ull;
  if (P < 64) mrow &= (1ull << P) - 1ull;
  uint64_t wmask = mrow;
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) wmask |= __shfl_xor(wmask, s, 64);
  if (lane == 0) wave_union[wave] = wmask;

  // Q^T fragments (B operand): row `col`, features kb*16 + 8*hh .. +7.
  u32x4 qf[KB];
  {
    // A lane past the block's rows reads the question's first kept row (the
    // item has at least one) and zeroes it, so all loads issue together.
    const int rr = row_ok ? r : 0;
    const bf16_t* qrow;
    if (kept_idx) {
      const int src = clampi(kept_idx[k0 + rr], 0, N - 1);
      qrow = qbase + ((size_t)b * N + src) * qstride + (size_t)h * D;
    } else {
      qrow = qbase + (size_t)(k0 + rr) * qstride + (size_t)h * D;
    }
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
      qf[kb] = *reinterpret_cast<const u32x4*>(qrow + kb * 16 + 8 * hh);
    // a negative scale is folded in here (bf16 sign flips), so the logits
    // below are always scaled by |scale|
    const uint32_t neg = (scale_log2 < 0.f) ? 0x80008000u : 0u;
    const uint32_t keep = row_ok ? 0xffffffffu : 0u;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) qf[kb] = (qf[kb] ^ neg) & keep;
    // Settle the query loads here: left pending, the compiler would wait for
    // them (vmcnt(0)) inside the tile loop, draining the prefetch ring.
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) asm volatile("" ::"v"(qf[kb]));
  }
  __syncthreads();
  uint64_t U = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) U |= wave_union[w];
  U = uniform64(U);
  wmask = uniform64(wmask);

  // Tile cursors over (adjacent passage, 64-token block): one for issuing
  // loads, one for computing.
  struct Cursor {
    uint64_t rem;
    int j, t, te;
  };
  auto advance = [&](Cursor& c) -> bool {
    if (c.j >= 0 && c.t + kTile < c.te) {
      c.t += kTile;
      return true;
    }
    while (c.rem) {
      const int j = __builtin_ctzll(c.rem);
      c.rem &= c.rem - 1ull;
      const int ts = __builtin_amdgcn_readfirstlane(p_ts[j]);
      const int te = __builtin_amdgcn_readfirstlane(p_te[j]);
      if (te > ts) {
        c.j = j; c.t = ts; c.te = te;
        return true;
      }
    }
    return false;
  };
  // Direct loads of one tile: instruction q fills LDS bytes [q*1024, +1024)
  // of the stage; lane l's 16 bytes are slot o = q*64 + l = (row, physical
  // chunk p).  K holds logical chunk p ^ (row % NCH) there, V holds logical
  // chunk p ^ vswz(row) (a key of row % 4 only, so the transposing reads of
  // tokens t, t+8, t+16, t+32 differ by constant offsets).  Rows past the
  // passage end re-read its last token (finite values, masked in the
  // softmax).
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  auto issue = [&](int stage, int t, int te) {
    bf16_t* Ks = Kbuf + stage * TILE;
    bf16_t* Vs = Vbuf + stage * TILE;
#pragma unroll
    for (int q = wave_s; q < NI; q += kLoaders) {
      const int o = q * 64 + lane;
      const int row = o / NCH, pch = o % NCH;
      const int ck = pch ^ (row & (NCH - 1));
      const int cv = pch ^ vswz(row);
      const int tok = min(t + row, te - 1);
      const size_t rowoff = ((size_t)tok * H + h) * D;
      lds_dma16(Kh + rowoff + ck * 8, lds_addr(Ks + q * 512));
      lds_dma16(Vh + rowoff + cv * 8, lds_addr(Vs + q * 512));
    }
  };

  f32x16_t acc[DT];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[t][v] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  // per-lane constants of the MFMA operand reads: K rows st*32 + col share
  // the swizzle key col % NCH; V^T reads follow the transposing-read layout
  const int g16 = lane >> 4, s16 = lane & 15;
  int koff[KB];                                       // K row col, chunk 2kb+hh
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
    koff[kb] = col * D + (((2 * kb + hh) ^ (col & (NCH - 1))) << 3);
  // V^T operand: token 4*hh + (s16 >> 2) (+ 16 per k-block, + 8 for the upper
  // half), feature 32*dt + 16*(g16 & 1) + 4*(s16 & 3)
  const int tr_tok = 4 * hh + (s16 >> 2);
  int voff[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    const int d = 32 * dt + 16 * (g16 & 1) + 4 * (s16 & 3);
    voff[dt] = tr_tok * D + (((d >> 3) ^ vswz(tr_tok)) << 3) + (d & 7);
  }

  // Matrix phase: O^T += V^T . P^T for the previous tile (weights pb/pl,
  // V tile in stage pv_stage), then S^T = K . Q^T for the tile in stage
  // s_stage into sacc.  NST (1 or 2) is the number of 32-token sub-tiles the
  // wave computes, starting at sub-tile sub0.
  f32x16_t sacc[2];
  u32x4 pb[4], pl[4];
  float acc_scale = 1.f;             // rescale of acc owed by the last softmax
  auto pv_product = [&](auto nst, int pv_stage) {
    constexpr int NST = decltype(nst)::value;
    __builtin_amdgcn_sched_barrier(0);
    if (__any(acc_scale != 1.f)) {   // some row's maximum moved
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[dt][v] *= acc_scale;
    }
    const bf16_t* Vs = Vbuf + pv_stage * TILE + sub0 * 32 * D;
#pragma unroll
    for (int hf = 0; hf < NST; ++hf) {
      u32x4 va[DT][2];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const bf16_t* vp = Vs + (32 * hf + 16 * g) * D + voff[dt];
          va[dt][g] = __builtin_shufflevector(ds_read_tr16(vp), ds_read_tr16(vp + 8 * D),
                                              0, 1, 2, 3);
        }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        acc[dt] = mfma32(va[dt][0], pb[2 * hf], acc[dt]);
        acc[dt] = mfma32(va[dt][1], pb[2 * hf + 1], acc[dt]);
        if (SPLIT_P) {
          acc[dt] = mfma32(va[dt][0], pl[2 * hf], acc[dt]);
          acc[dt] = mfma32(va[dt][1], pl[2 * hf + 1], acc[dt]);
        }
      }
    }
    // Schedule: sixteen V^T reads ahead, then one MFMA (two with the split
    // weights) per two reads, so the read latency hides behind the matrix
    // pipe (left alone, the compiler waits for every operand pair in turn).
    {
      constexpr int R = NST * 4 * DT;
      constexpr int MPS = SPLIT_P ? 2 : 1;
      constexpr int M = NST * 2 * DT * MPS;
      constexpr int PRE = R < 16 ? R : 16;
      constexpr int STEPS = (R - PRE) / 2;
      __builtin_amdgcn_sched_group_barrier(0x100, PRE, 0);   // LDS reads
#pragma unroll
      for (int i = 0; i < STEPS; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, MPS, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, M - STEPS * MPS, 0);
    }
  };
  auto s_product = [&](auto nst, int s_stage) {
    constexpr int NST = decltype(nst)::value;
    __builtin_amdgcn_sched_barrier(0);
    const bf16_t* Ks = Kbuf + s_stage * TILE + sub0 * 32 * D;
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      u32x4 ka[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        ka[kb] = *reinterpret_cast<const u32x4*>(Ks + st * 32 * D + koff[kb]);
#pragma unroll
      for (int v = 0; v < 16; ++v) sacc[st][v] = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) sacc[st] = mfma32(ka[kb], qf[kb], sacc[st]);
    }
    // Schedule: eight K reads ahead (all of them for one sub-tile at d_h 64),
    // then one MFMA per read.
    {
      constexpr int R = NST * KB;
      constexpr int PRE = R < 8 ? R : 8;
      __builtin_amdgcn_sched_group_barrier(0x100, PRE, 0);
#pragma unroll
      for (int i = 0; i < R - PRE; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, PRE, 0);
    }
  };
  // Vector phase: online softmax over the scores of this lane's row in sacc
  // (sub-tiles with `full`, `rem`, adjacency bias `mbias`); rescales acc and
  // leaves the bf16 weights in pb (and their remainders in pl).
  auto softmax = [&](auto nst, bool full, int rem, float mbias) {
    constexpr int NST = decltype(nst)::value;
    __builtin_amdgcn_sched_barrier(0);
    // (a negative scale was folded into the query fragments: c > 0)
    const float c = fabsf(scale_log2);
    if (!full) {                     // tokens past the passage end
      // kept as a branch: selecting on every tile would cost 64 VALU ops
      asm volatile("");
#pragma unroll
      for (int st = 0; st < NST; ++st)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (32 * st + 8 * (v >> 2) + (v & 3) >= rem) sacc[st][v] = -INFINITY;
    }
    float sm = sacc[0][0];
#pragma unroll
    for (int st = 0; st < NST; ++st)
#pragma unroll
      for (int v = 0; v < 16; ++v) sm = fmaxf(sm, sacc[st][v]);
    sm = fmaxf(sm, swap_halves(sm));
    const float mt = (sm == -INFINITY) ? -INFINITY : fmaf(sm, c, mbias);
    const float m_new = fmaxf(m_run, mt);
    const float alpha = (m_new == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run - m_new);
    const float bias = mbias - ((m_new == -INFINITY) ? 0.f : m_new);
    m_run = m_new;
    float ls = 0.f;
#pragma unroll
    for (int kb2 = 0; kb2 < 2 * NST; ++kb2) {
      float pv[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // scores are finite on a full tile (a row not adjacent to the
        // passage has bias -inf); past the passage end the weight is 0
        const float x = sacc[kb2 >> 1][8 * (kb2 & 1) + e];
        pv[e] = __builtin_amdgcn_exp2f(fmaf(x, c, bias));   // 0 for a masked token
        ls += pv[e];
      }
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) w[q] = pack2_bf16(pv[2 * q], pv[2 * q + 1]);
      pb[kb2] = u32x4{w[0], w[1], w[2], w[3]};
      if (SPLIT_P) {
        uint32_t wl[4];
#pragma unroll
        for (int q = 0; q < 4; ++q)
          wl[q] = pack2_bf16(pv[2 * q] - __uint_as_float(w[q] << 16),
                             pv[2 * q + 1] - __uint_as_float(w[q] & 0xffff0000u));
        pl[kb2] = u32x4{wl[0], wl[1], wl[2], wl[3]};
      }
    }
    l_run = l_run * alpha + ls;
    acc_scale = alpha;               // applied before the next PV product
  };

  // Tile loop, two half-steps per tile separated by barriers: the matrix
  // phase of tile i (PV of tile i-1, S of tile i), then its softmax.  Group B
  // (waves 4-7) takes one extra barrier first, so it runs half a step behind
  // group A (waves 0-3): on each SIMD one wave's matrix work overlaps the
  // other's vector work.  Group A issues and awaits every tile load; a tile
  // is awaited before the barrier that precedes its first use by either
  // group.  Tiles i-1 and i stay in use until group B's step i ends, so loads
  // run STAGES-2 tiles ahead.
  const bool group_b = wave >= 4;
  const bool busy = wmask != 0;
  Cursor ci{U, -1, 0, 0}, cc{U, -1, 0, 0};
  int issued = 0;
  if (!group_b) {
#pragma unroll
    for (int s = 0; s < kStages - 2; ++s)
      if (advance(ci)) { issue(issued % kStages, ci.t, ci.te); ++issued; }
  } else {
    barrier_nofence();
  }
  // tile i's loads have landed once at most `ahead` later tiles are pending
  auto wait_tile = [&](int ahead) {
    if (ahead >= 2) wait_vmem<2 * LPT>();
    else if (ahead == 1) wait_vmem<LPT>();
    else wait_vmem<0>();
  };
  // Step i: PV of tile i-1 (zero weights at i = 0), S and softmax of tile i;
  // a final step past the last tile does only the PV.
  auto busy_loop = [&](auto nst) {
    // The first matrix phase adds tile 0's V with zero weights (exactly 0).
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      pb[q] = u32x4{0u, 0u, 0u, 0u};
      pl[q] = u32x4{0u, 0u, 0u, 0u};
    }
    int prev_stage = 0;
    for (int i = 0;; ++i) {
      const bool more = advance(cc);
      if (!more && i == 0) break;
      if (more) {
        if (!group_b) wait_tile(issued - i - 1);
        barrier_nofence();
        if (!group_b && advance(ci)) { issue(issued % kStages, ci.t, ci.te); ++issued; }
      }
      pv_product(nst, prev_stage);
      if (!more) break;
      const int stage = i % kStages;
      s_product(nst, stage);
      barrier_nofence();
      // accumulator element v of sub-tile st is token 32*st + 8*(v/4) + v%4
      // + 4*hh of the wave's first sub-tile; it exists if that is below rem
      const int t0 = cc.t + 32 * sub0;
      softmax(nst, t0 + 32 * decltype(nst)::value <= cc.te, cc.te - t0 - 4 * hh,
              ((mrow >> cc.j) & 1ull) ? 0.f : -INFINITY);
      prev_stage = stage;
    }
  };
  if (!busy) {
    // A wave without kept rows only keeps step with the barriers (and, in
    // group A, streams its share of the tiles).
    for (int i = 0; advance(cc); ++i) {
      if (!group_b) wait_tile(issued - i - 1);
      barrier_nofence();
      if (!group_b && advance(ci)) { issue(issued % kStages, ci.t, ci.te); ++issued; }
      barrier_nofence();
    }
  } else if (split) {
    busy_loop(IntC<1>{});
  } else {
    busy_loop(IntC<2>{});
  }
  if (!group_b) barrier_nofence();

  // Merge the two halves of a split block (online-softmax combination):
  // the upper half's wave hands (acc, m, l) over through the LDS ring.
  if (any_split) {
    __syncthreads();                 // every wave is done with the ring
    // a pair's slot: blocks 0/1 (1-2 blocks) or 4/5 (5-6 blocks) use slots 0/1
    float* xb = reinterpret_cast<float*>(Kbuf) + (wb & 1) * (DT * 16 + 2) * 64;
    const bool paired = split && wb < nrb;   // waves past the last block hold no rows
    if (paired && half == 1) {
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v) xb[(dt * 16 + v) * 64 + lane] = acc[dt][v];
      xb[(DT * 16) * 64 + lane] = m_run;
      xb[(DT * 16 + 1) * 64 + lane] = l_run;
    }
    __syncthreads();
    if (paired && half == 1) return;
    if (paired) {
      const float m1 = xb[(DT * 16) * 64 + lane];
      const float l1 = xb[(DT * 16 + 1) * 64 + lane];
      const float M = fmaxf(m_run, m1);
      const float a0 = (m_run == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m_run - M);
      const float a1 = (m1 == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(m1 - M);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          acc[dt][v] = acc[dt][v] * a0 + xb[(dt * 16 + v) * 64 + lane] * a1;
      l_run = l_run * a0 + l1 * a1;
      m_run = M;
    }
  }

  // finalize
  const float l_tot = l_run + swap_halves(l_run);
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
    const int RB = (p.k_max + kMaxRows - 1) / kMaxRows;
    const int n_items = p.B * p.H * RB;
    const int grid = ((n_items + 7) / 8) * 8;
    const float sl2 = p.sm_scale * kLog2e;
#define SKIP_ATTN_BF16(DD, SP)                                                               \
  hipLaunchKernelGGL((attn_bf16_kernel<DD, SP>), dim3(grid), dim3(kThreads), 0, s,           \
                     (const bf16_t*)q.base, q.kept_idx, q.N, qstride, kept_offsets,          \
                     (const bf16_t*)Kh, (const bf16_t*)Vh, passage_offsets, query_passages,  \
                     rowmask, p.H, p.total_kept, p.total_passages, p.total_tokens, p.k_max,  \
                     p.P_max, RB, n_items, sl2, O, p.o_f32, lse)
    // float32 output: split softmax weights (bf16 hi + lo) for near-fp32 accuracy
    if (p.d_h == 64) {
      if (p.o_f32) SKIP_ATTN_BF16(64, true);
      else SKIP_ATTN_BF16(64, false);
    } else {
      if (p.o_f32) SKIP_ATTN_BF16(128, true);
      else SKIP_ATTN_BF16(128, false);
    }
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

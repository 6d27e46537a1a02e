// Sparse cross-attention restricted to the bipartite graph (paper App. B.3,
// Def. B.3 attention rule; Alg. 1, fuse step).
//
// For kept row i of question b and head h, the logits run over every token of
// every passage adjacent to i (one 64-bit neighbour mask per row):
//   e_m = sm_scale * <Qh[i,h], Kh[m,h]>,  O = softmax(e) . Vh,  LSE = log sum exp e.
//
// bf16 path (MFMA): passage-major, only the graph's edges are computed (the
// kernel comment below); a device-built work list orders the items by cost.
//
// fp32 path: one wave per (kept row, head); 64 tokens per step, lane = token
// for the logits, lane = feature for the PV product.
#include "skip_common.h"
#include "skip_internal.h"
#include "skip_plan.h"

namespace skip {

typedef short s16x4_t __attribute__((ext_vector_type(4)));
template <int N>
struct IntC {                     // a compile-time count passed to a generic lambda
  static constexpr int value = N;
};
// f(IntC<0>), .., f(IntC<N-1>)
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(IntC<I>{});
    static_for<N, I + 1>(f);
  }
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Value of lane l ^ 32 (v_permlane32_swap: the two half-waves trade places).
__device__ __forceinline__ float swap_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                  false, false);
  return __uint_as_float(__lane_id() < 32 ? r[1] : r[0]);
}

// Value of lane l ^ 16 (v_permlane16_swap: odd and even 16-lane rows trade).
__device__ __forceinline__ float swap16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x),
                                                  false, false);
  return __uint_as_float((__lane_id() & 16) ? r[0] : r[1]);
}

// Transposing LDS read (ds_read_b64_tr_b16) at byte address lds + OFF: in
// each group of 16 lanes, lane j receives element j & 3 of the 8-byte pieces
// addressed by lanes (j >> 2) + 4e, e = 0..3.  Issued through inline
// assembly so that the constant offset sits in the instruction (the builtin
// takes a full address per read); the compiler does not track its
// completion, so the results pass through lds_wait_all before any use.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
template <int OFF>
__device__ __forceinline__ u32x2 ds_read_tr16_at(uint32_t lds) {
  static_assert(OFF >= 0 && OFF < 65536 && OFF % 8 == 0, "DS offset field");
  u32x2 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(lds), "i"(OFF));
  return r;
}

// Waits for every outstanding LDS read of the wave; the registers passed
// through it are the values after the wait (a true dependency for the
// compiler, so no use of them is scheduled above it).
template <int N>
__device__ __forceinline__ void lds_wait_all(u32x2 (&v)[N]) {
  static_assert(N == 16 || N == 8, "operand count");
  if constexpr (N == 16) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]),
                   "+v"(v[6]), "+v"(v[7]), "+v"(v[8]), "+v"(v[9]), "+v"(v[10]), "+v"(v[11]),
                   "+v"(v[12]), "+v"(v[13]), "+v"(v[14]), "+v"(v[15])
                 :
                 : "memory");
  } else {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]), "+v"(v[4]), "+v"(v[5]),
                   "+v"(v[6]), "+v"(v[7])
                 :
                 : "memory");
  }
}

// ---------------------------------------------------------------------------
// bf16 path, passage-major.  Attention is computed only on the graph's edges:
// for each passage j, only the kept rows adjacent to j (Def. B.3: a row's
// softmax runs over the tokens of its neighbour passages, and no other pair
// is touched), so the work grows with the number of edges and a passage
// adjacent to none of an item's rows is never read.
//
// Work item = (question b, head h, chunk of <= kSpRows kept rows).  The item
// walks the passages with at least one adjacent row in the chunk, in
// ascending order, 32 tokens at a time.  K and V tiles of head h stream
// through two LDS rings of three tiles, one barrier per tile; two loader
// waves (one for K, one for V) keep four more tiles in flight in registers
// and write each into the ring when its slot frees.  For each passage the
// adjacent rows (a 192-bit row mask per passage) form blocks of 16 in row
// order; compute wave w takes blocks w and w + 6.  Per tile and block:
//   S^T (32 tokens x 16 rows) = K_tile . Q^T        v_mfma_f32_16x16x32_bf16
//   online softmax in fp32 (base 2); each weight p split into bf16 hi + lo
//   (hi = p truncated, lo = the rest rounded), so the PV product sees p to
//   about 2^-16 relative and the result does not depend on the output type,
//   O^T (d_h x 16 rows)     += V_tile^T . (P_hi + P_lo)^T
// Computing the transposed products keeps each query row in one lane column
// (row statistics need an exchange among the four lanes of that column) and
// makes the S^T accumulator the P^T operand; V^T comes from transposing LDS
// reads in the token order of that layout.  The queries of a block's rows
// sit in registers, loaded at the previous busy passage's last tile.  After
// a passage's last tile each block's partial (O, max, sum) is merged into
// the item's accumulators, fp32 in LDS for every row of the chunk, by
// log-sum-exp rescaling; one passage's blocks hold disjoint rows and
// passages merge in ascending order (a barrier at least between two), so the
// result is deterministic.  The item ends by writing O = acc / sum and LSE
// for every row of the chunk (0 and -inf for a row without neighbours).
constexpr int kSpTile = 32;               // tokens per K/V tile
constexpr int kSpStages = 3;              // K (and V) tiles resident in LDS
constexpr int kSpRegTiles = 4;            // K (and V) tiles in flight in loader registers
constexpr int kSpCompute = kSpRows / 32;  // compute waves (two 16-row blocks each)
constexpr int kSpWaves = kSpCompute + 2;  // + a K loader and a V loader
constexpr int kSpThreads = 64 * kSpWaves;
constexpr float kLazy = 8.f;              // log2 slack of the softmax reference maximum
static_assert(kSpRows <= 3 * 64, "row masks have three 64-bit words");

// Position of the n-th (from 0) set bit of x; n < popcount(x).
__device__ __forceinline__ int nth_bit64(uint64_t x, int n) {
  int pos = 0;
#pragma unroll
  for (int w = 32; w >= 1; w >>= 1) {
    const int c = __popcll(x & ((1ull << w) - 1ull));
    if (n >= c) {
      n -= c;
      x >>= w;
      pos += w;
    }
  }
  return pos;
}

// Work item record: {question, first kept row (global), first passage,
// head | rows << 8 | passages << 16}; question -1: no item.
template <int D>
__global__ void __launch_bounds__(kSpThreads)
attn_sparse_kernel(const bf16_t* __restrict__ qbase, const int32_t* __restrict__ kept_idx,
                   int N, int qstride, const bf16_t* __restrict__ Kh,
                   const bf16_t* __restrict__ Vh, const int32_t* __restrict__ passage_offsets,
                   const uint64_t* __restrict__ rowmask, const int4* __restrict__ items, int H,
                   int total_tokens, float scale_log2, void* __restrict__ O, int o_f32,
                   float* __restrict__ lse) {
  constexpr int NCH = D / 8;               // 16-byte chunks per token row
  constexpr int NC4 = D / 4;               // 4-float chunks per accumulator row
  constexpr int KB = D / 32;               // k-blocks of QK^T (32 features each)
  constexpr int DB = D / 16;               // 16-wide feature blocks of O
  // Tiles are token-major with padded rows: K rows of D + 8 elements put the
  // sixteen tokens of one S^T operand read on distinct banks, V rows of D +
  // 16 the sixteen tokens of one transposing read (two 8-byte pieces each);
  // every operand read is then a register base plus an immediate offset.
  constexpr int SK = D + 8, SV = D + 16;   // row strides (elements)
  constexpr int TK = kSpTile * SK, TV = kSpTile * SV;
  constexpr int NI = kSpTile * NCH / 64;   // 16-byte loads per lane per K (or V) tile
  __shared__ __attribute__((aligned(1024))) bf16_t Kbuf[kSpStages * TK];
  __shared__ __attribute__((aligned(1024))) bf16_t Vbuf[kSpStages * TV];
  __shared__ __attribute__((aligned(16))) float Oacc[kSpRows * D];
  __shared__ float m_acc[kSpRows], l_acc[kSpRows];
  __shared__ uint64_t rmask[3][kSpMaxP];   // rows 64w..64w+63 adjacent to each passage
  __shared__ int p_ts[kSpMaxP], p_te[kSpMaxP], p_cnt[kSpMaxP];
  __shared__ int32_t qsrc[kSpRows];        // visual-token index of each row (fused route)

  const int4 item = items[blockIdx.x];
  const int b = item.x;
  if (b < 0) return;
  const int row0 = item.y, p0 = item.z;
  const int h = item.w & 0xff;
  const int nrows = (item.w >> 8) & 0xff;
  const int P = (item.w >> 16) & 0xff;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave

  // accumulators, passage ranges, row sources, row masks per passage
  const uint64_t pm = (P >= 64) ? ~0ull : ((1ull << P) - 1ull);
  const uint64_t mk = (tid < nrows) ? (rowmask[row0 + tid] & pm) : 0ull;
  const int src = (kept_idx && tid < nrows) ? kept_idx[row0 + tid] : 0;
  int ts = 0, te = 0;
  if (tid < P) range_of(passage_offsets, p0 + tid, total_tokens, ts, te);
  for (int i = tid; i < nrows * NC4; i += kSpThreads)
    reinterpret_cast<float4*>(Oacc)[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  if (tid < nrows) {
    m_acc[tid] = -INFINITY;
    l_acc[tid] = 0.f;
    qsrc[tid] = clampi(src, 0, N - 1);
  }
  if (tid < P) {
    p_ts[tid] = ts;
    p_te[tid] = te;
  }
  if (wave < 3) {
    for (int j = 0; j < P; ++j) {
      const uint64_t bal = __ballot((mk >> j) & 1ull);
      if (lane == 0) rmask[wave][j] = bal;
    }
  }
  __syncthreads();
  if (tid < P) p_cnt[tid] = __popcll(rmask[0][tid]) + __popcll(rmask[1][tid]) +
                            __popcll(rmask[2][tid]);
  __syncthreads();
  // passages with at least one adjacent row of the chunk (and some tokens)
  const bool touched = lane < P && p_cnt[lane] > 0 && p_te[lane] > p_ts[lane];
  const uint64_t U = uniform64(__ballot(touched));

  // Tile cursor over (touched passage, 32-token block).
  struct Cursor {
    uint64_t rem;
    int j, t, ts, te;
  };
  auto advance = [&](Cursor& cu) -> bool {
    if (cu.j >= 0 && cu.t + kSpTile < cu.te) {
      cu.t += kSpTile;
      return true;
    }
    if (!cu.rem) return false;
    const int j = __builtin_ctzll(cu.rem);
    cu.rem &= cu.rem - 1ull;
    cu.j = j;
    cu.ts = __builtin_amdgcn_readfirstlane(p_ts[j]);
    cu.te = __builtin_amdgcn_readfirstlane(p_te[j]);
    cu.t = cu.ts;
    return true;
  };

  // One barrier per tile publishes it; the loads run two tiles ahead.
  int n_tiles = 0;
  for (uint64_t r = U; r; r &= r - 1ull) {
    const int j = __builtin_ctzll(r);
    n_tiles += (__builtin_amdgcn_readfirstlane(p_te[j]) - __builtin_amdgcn_readfirstlane(p_ts[j]) +
                kSpTile - 1) / kSpTile;
  }

  if (wave >= kSpCompute) {
    // ---- loader waves: the first streams K, the second V --------------------
    // (their LDS writes must land before each barrier; issuing ahead of the
    // compute waves' operand reads keeps them from queueing behind those)
    __builtin_amdgcn_s_setprio(3);
    const bool isV = wave == kSpCompute + 1;
    const bf16_t* gsrc = isV ? Vh : Kh;
    bf16_t* buf = isV ? Vbuf : Kbuf;
    const int S = isV ? SV : SK, T = isV ? TV : TK;
    // load q of a tile: lane l takes 16-byte chunk (q*64 + l) % NCH of token
    // row (q*64 + l) / NCH; byte offsets from the tile's first token
    uint32_t voff[NI];
#pragma unroll
    for (int q = 0; q < NI; ++q) {
      const int o = q * 64 + lane;
      voff[q] = (uint32_t)(((o / NCH) * H * D + (o % NCH) * 8) * 2);
    }
    const int lds_lane = (lane / NCH) * S + (lane % NCH) * 8;
    const bf16_t* hsrc = gsrc + (size_t)h * D;
    // Tiles travel through registers: global loads run kSpRegTiles tiles
    // ahead of the LDS ring (which holds the tile being consumed and the next
    // one), so the loads keep streaming while the compute waves merge or
    // start a passage.  Slot n % kSpRegTiles holds tile n.
    u32x4 rg[kSpRegTiles][NI];
    auto gload = [&](auto slot, int t, int te_) {
      const bf16_t* tbase = hsrc + (size_t)t * H * D;
      const int over_base = t - (te_ - 1);
#pragma unroll
      for (int q = 0; q < NI; ++q) {
        // rows past the passage's end read its last token (finite values,
        // masked in the softmax)
        const int row = (q * 64 + lane) / NCH;
        const uint32_t o = voff[q] - (uint32_t)(max(over_base + row, 0) * H * D * 2);
        rg[decltype(slot)::value][q] = *reinterpret_cast<const u32x4*>(
            reinterpret_cast<const char*>(tbase) + o);
      }
      // tiles issue in order (the wait counts assume it)
      asm volatile("" ::: "memory");
    };
    auto swrite = [&](auto slot, int n) {
      bf16_t* dst = buf + (n % kSpStages) * T + lds_lane;
#pragma unroll
      for (int q = 0; q < NI; ++q)
        *reinterpret_cast<u32x4*>(dst + q * (64 / NCH) * S) = rg[decltype(slot)::value][q];
    };
    // Every step issues one tile's loads, unconditionally (past the last
    // tile the cursor stays put and the last tile is read again), so that
    // the compiler's wait counts before each register slot's LDS write are
    // exact: the slot's loads are the oldest of the four in flight.
    Cursor ci{U, -1, 0, 0, 0};
    auto issue = [&](auto slot) {
      advance(ci);
      gload(slot, ci.t, ci.te);
    };
    static_assert(kSpRegTiles == 4 && kSpStages == 3, "slot arithmetic below");
    if (n_tiles > 0) {
      // prologue: loads of tiles 0 .. 3, tiles 0 and 1 into LDS, loads of
      // tiles 4 and 5
      issue(IntC<0>{});
      issue(IntC<1>{});
      issue(IntC<2>{});
      issue(IntC<3>{});
      swrite(IntC<0>{}, 0);
      issue(IntC<0>{});
      swrite(IntC<1>{}, 1);            // (a repeat of tile 0 if there is one tile)
      issue(IntC<1>{});
      // step i: after its barrier the LDS slot of tile i-1, which every wave
      // finished in step i-1, is free; tile i+2 goes there from register slot
      // (i+2) % 4, which then takes tile i+6
      auto step = [&](auto u, int i) {
        constexpr int sl = (decltype(u)::value + 2) % kSpRegTiles;
        if (i < n_tiles) {
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // tiles <= i+1 written
          barrier_nofence();                                     // tile i is published
          // (past the last tile a repeat, into a slot that is not read again)
          swrite(IntC<sl>{}, i + 2);
        }
        issue(IntC<sl>{});
      };
      // whole groups of four steps, one exit: the loads of every step are
      // unconditional, so each slot's wait count is the same on every path
      for (int i = 0; i < n_tiles; i += kSpRegTiles) {
        step(IntC<0>{}, i);
        step(IntC<1>{}, i + 1);
        step(IntC<2>{}, i + 2);
        step(IntC<3>{}, i + 3);
      }
    }
  } else {
    // ---- compute waves ------------------------------------------------------
    // Lane layout of every product (16 x 16 blocks): r16 = lane & 15 is the
    // lane's row within a block (the column of S^T, P^T and O^T); g = lane
    // >> 4 picks tokens 4g..4g+3 of each 16-token half of S^T, the k-slice
    // 8g..8g+7 of P^T (those same eight tokens, halves in order) and
    // features 16db + 4g..4g+3 of O^T.
    const int g = lane >> 4;
    const int r16 = lane & 15;
    // K (A of S^T): token r16 (+16), features 32kb + 8g .. +7
    const int koff = r16 * SK + 8 * g;
    // V^T (A of O^T) by transposing reads: lane (e = r16 >> 2, q = r16 & 3)
    // addresses token 4g + e (+16), features 16db + 4q .. +3; lane r16 then
    // holds feature 16db + r16 of tokens 4g .. 4g+3
    const uint32_t vlds = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)(
        Vbuf + (4 * g + (r16 >> 2)) * SV + 4 * (r16 & 3));
    // a negative scale is folded into the queries (bf16 sign flips), so the
    // logits are scaled by |scale| and their maximum is a plain maximum
    const uint32_t neg = (scale_log2 < 0.f) ? 0x80008000u : 0u;
    const float sc = fabsf(scale_log2);
    // Touched passages in which this wave has its first block (block `wave`)
    // and its second (block wave + kSpCompute).
    const uint64_t bmask = uniform64(
        __ballot(lane < P && ((U >> lane) & 1ull) && p_cnt[lane] > 16 * wave));
    const uint64_t bmask2 = uniform64(__ballot(
        lane < P && ((U >> lane) & 1ull) && p_cnt[lane] > 16 * (wave + kSpCompute)));
    // Queries of the blocks' rows go straight into qf.  For the wave's busy
    // passages in order: at the first tile of busy passage k the lookup of
    // busy passage k+1 starts and runs in phases, one per step: (1) the
    // passage's row masks, (2) this lane's rows (the n-th adjacent row, n =
    // 16 * block + r16) and their visual-token indices.  At passage k's last
    // tile, once its S^T products have read qf, the lookup is finished and
    // the loads of passage k+1's queries are issued into qf; they land while
    // that tile's softmax, PV product and merge run.  A lane past a block's
    // rows loads a placeholder row, whose scores land in a column that is
    // never merged.
    u32x4 qf[2][KB];
    int lk_j = -1, lk_phase = 2;       // passage being looked up; phases done (2: done)
    uint64_t lkw0 = 0, lkw1 = 0, lkw2 = 0;
    int lk_row[2] = {-1, -1}, lk_src[2] = {0, 0};   // result of the lookup
    int nx_row[2] = {-1, -1};          // rows of the queries in qf for the next passage
    auto nth_row = [&](int n) -> int {
      const int c0 = __popcll(lkw0), c1 = __popcll(lkw1), c2 = __popcll(lkw2);
      if (n >= c0 + c1 + c2) return -1;
      if (n < c0) return nth_bit64(lkw0, n);
      if (n < c0 + c1) return 64 + nth_bit64(lkw1, n - c0);
      return 128 + nth_bit64(lkw2, n - c0 - c1);
    };
    auto lookup_phase = [&]() {
      if (lk_phase == 0) {
        lkw0 = uniform64(rmask[0][lk_j]);
        lkw1 = uniform64(rmask[1][lk_j]);
        lkw2 = uniform64(rmask[2][lk_j]);
      } else {
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          lk_row[k] = nth_row(16 * (wave + k * kSpCompute) + r16);
          lk_src[k] = kept_idx ? qsrc[lk_row[k] >= 0 ? lk_row[k] : 0] : 0;
        }
      }
      ++lk_phase;
    };
    auto start_lookup = [&](int j) {   // j < 0: nothing
      lk_j = j;
      lk_phase = j < 0 ? 2 : 0;
    };
    // qf <- the queries of the looked-up passage's rows (its second block
    // only where this wave has one)
    auto load_q = [&]() {
      if (lk_j < 0) return;
      while (lk_phase < 2) lookup_phase();
      const bool two_next = (bmask2 >> lk_j) & 1ull;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        if (k == 1 && !two_next) break;
        nx_row[k] = lk_row[k];
        const int rr = lk_row[k] >= 0 ? lk_row[k] : 0;
        const bf16_t* qrow = kept_idx
            ? qbase + ((size_t)b * N + lk_src[k]) * qstride + (size_t)h * D
            : qbase + (size_t)(row0 + rr) * qstride + (size_t)h * D;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
          qf[k][kb] = *reinterpret_cast<const u32x4*>(qrow + 32 * kb + 8 * g);
      }
    };
    start_lookup(bmask ? __builtin_ctzll(bmask) : -1);
    load_q();

    // per block: row of this lane's column, O^T partial, running maximum and
    // row sum of the weights (per lane until the merge)
    int acc_row[2] = {-1, -1};
    f32x4_t acc[2][DB];
    float m_run[2], l_run[2];

    // a block's partial into the item's accumulators
    auto merge = [&](auto kk) {
      constexpr int k = decltype(kk)::value;
      float l_tot = l_run[k] + swap16(l_run[k]);
      l_tot += swap_halves(l_tot);
      const int ri = acc_row[k];
      if (ri < 0) return;
      const float mo = m_acc[ri], lo = l_acc[ri];
      float4* orow = reinterpret_cast<float4*>(Oacc + ri * D);
      const float mn = fmaxf(mo, m_run[k]);
      const float a = __builtin_amdgcn_exp2f(mo - mn);    // 0 while the row is empty
      const float cb = __builtin_amdgcn_exp2f(m_run[k] - mn);
      float4 ov[DB];                    // features 16db + 4g .. +3
#pragma unroll
      for (int db = 0; db < DB; ++db) ov[db] = orow[(4 * db + g) ^ (ri & (NC4 - 1))];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        float4 o = ov[db];
        o.x = fmaf(o.x, a, acc[k][db][0] * cb);
        o.y = fmaf(o.y, a, acc[k][db][1] * cb);
        o.z = fmaf(o.z, a, acc[k][db][2] * cb);
        o.w = fmaf(o.w, a, acc[k][db][3] * cb);
        orow[(4 * db + g) ^ (ri & (NC4 - 1))] = o;
      }
      if (g == 0) {
        m_acc[ri] = mn;
        l_acc[ri] = fmaf(lo, a, l_tot * cb);
      }
    };

    // One tile for block K0: S^T = K . Q^T (two 16-token halves), online
    // softmax of each row, O^T += V^T . P^T.  All of a phase's LDS reads are
    // issued before its products (the V reads before the softmax, which
    // hides them).  A wave with two blocks in the passage runs them one
    // after the other.
    auto tile = [&](auto k0, int stage, int t, int te_, bool first) {
      constexpr int K0 = decltype(k0)::value;
      constexpr int NBK = 1;
      if (first) {
#pragma unroll
        for (int k = 0; k < NBK; ++k) {
#pragma unroll
          for (int db = 0; db < DB; ++db) acc[K0 + k][db] = f32x4_t{0.f, 0.f, 0.f, 0.f};
          m_run[K0 + k] = -INFINITY;
          l_run[K0 + k] = 0.f;
        }
      }
      const bf16_t* Ks = Kbuf + stage * TK + koff;
      u32x4 ka[2][KB];
#pragma unroll
      for (int th = 0; th < 2; ++th)
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
          ka[th][kb] = *reinterpret_cast<const u32x4*>(Ks + th * 16 * SK + 32 * kb);
      __builtin_amdgcn_sched_barrier(0);
      f32x4_t s[NBK][2];
#pragma unroll
      for (int k = 0; k < NBK; ++k)
#pragma unroll
        for (int th = 0; th < 2; ++th) {
          s[k][th] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kb = 0; kb < KB; ++kb) s[k][th] = mfma16_bf16(ka[th][kb], qf[K0 + k][kb], s[k][th]);
        }
      __builtin_amdgcn_sched_barrier(0);
      // V reads (DB feature blocks x two 16-token halves) at constant offsets
      // from one address
      const uint32_t vaddr = vlds + (uint32_t)(stage * TV * 2);
      u32x2 vr[2 * DB];
      static_for<2 * DB>([&](auto c) {
        constexpr int th = decltype(c)::value & 1, db = decltype(c)::value >> 1;
        vr[2 * db + th] = ds_read_tr16_at<(th * 16 * SV + 16 * db) * 2>(vaddr);
      });
      __builtin_amdgcn_sched_barrier(0);
      // Online softmax of this lane's row: s[k][th][j] is token 16th + 4g + j
      // of the tile.  The weights are taken against a reference maximum m_run
      // that moves only when a tile's maximum exceeds it by more than 2^kLazy
      // (the weights then stay <= 2^kLazy and acc is rescaled only then, not
      // on every tile).
      u32x4 pb[NBK], pl[NBK];
#pragma unroll
      for (int k = 0; k < NBK; ++k) {
        if (t + kSpTile > te_) {
          const int rem = te_ - t - 4 * g;        // tokens 4g + j < rem are valid
#pragma unroll
          for (int th = 0; th < 2; ++th)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              if (16 * th + j >= rem) s[k][th][j] = -INFINITY;
        }
        // this lane's 8 logits; the row maximum (over the four lanes of the
        // row) is needed only when some row's reference has to move, which
        // a lane can tell from its own logits
        const float lm = fmaxf(fmaxf(fmaxf(s[k][0][0], s[k][0][1]), fmaxf(s[k][0][2], s[k][0][3])),
                               fmaxf(fmaxf(s[k][1][0], s[k][1][1]), fmaxf(s[k][1][2], s[k][1][3])));
        float m_new = m_run[K0 + k];                        // -inf on a block's first tile
        if (__any(lm * sc > m_new + kLazy)) {
          float sm = fmaxf(lm, swap16(lm));
          sm = fmaxf(sm, swap_halves(sm));
          const float tmax = sm * sc;                       // the tile has a valid token
          if (tmax > m_new + kLazy) {
            // acc and the sum are 0 before a block's first tile: nothing to
            // rescale then
            const float alpha = m_new != -INFINITY ? __builtin_amdgcn_exp2f(m_new - tmax) : 1.f;
            m_new = tmax;
            l_run[K0 + k] *= alpha;
#pragma unroll
            for (int db = 0; db < DB; ++db) acc[K0 + k][db] *= alpha;
          }
          m_run[K0 + k] = m_new;
        }
        // each weight p as a bf16 pair hi + lo: hi = p truncated to bf16 (its
        // top 16 bits, v_perm_b32 packs two), lo = the rest p - hi (exact)
        // rounded to bf16, so hi + lo is p to about 2^-16 relative
        uint32_t w[4], wl[4];
        float ls = 0.f;
#pragma unroll
        for (int th = 0; th < 2; ++th)
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const float p0 = __builtin_amdgcn_exp2f(fmaf(s[k][th][2 * q], sc, -m_new));
            const float p1 = __builtin_amdgcn_exp2f(fmaf(s[k][th][2 * q + 1], sc, -m_new));
            ls += p0 + p1;
            const uint32_t b0 = __float_as_uint(p0), b1 = __float_as_uint(p1);
            w[2 * th + q] = __builtin_amdgcn_perm(b1, b0, 0x07060302u);
            wl[2 * th + q] = pack2_bf16(p0 - __uint_as_float(b0 & 0xffff0000u),
                                        p1 - __uint_as_float(b1 & 0xffff0000u));
          }
        pb[k] = u32x4{w[0], w[1], w[2], w[3]};
        pl[k] = u32x4{wl[0], wl[1], wl[2], wl[3]};
        l_run[K0 + k] += ls;
      }
      __builtin_amdgcn_sched_barrier(0);
      // O^T += V^T . P^T
      lds_wait_all(vr);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const u32x4 va = __builtin_shufflevector(vr[2 * db], vr[2 * db + 1], 0, 1, 2, 3);
#pragma unroll
        for (int k = 0; k < NBK; ++k) {
          acc[K0 + k][db] = mfma16_bf16(va, pb[k], acc[K0 + k][db]);
          acc[K0 + k][db] = mfma16_bf16(va, pl[k], acc[K0 + k][db]);
        }
      }
    };

    Cursor cc{U, -1, 0, 0, 0};
    for (int i = 0; i < n_tiles; ++i) {
      advance(cc);
      const bool busy = (bmask >> cc.j) & 1ull;
      const bool two = (bmask2 >> cc.j) & 1ull;
      const bool first = cc.t == cc.ts;
      const bool last = cc.t + kSpTile >= cc.te;   // the passage's last tile
      if (busy && first) {
        // this passage's queries are in qf (a negative scale's sign folded
        // in here); the lookup of the next busy passage starts
        acc_row[0] = nx_row[0];
        acc_row[1] = nx_row[1];
        if (neg) {
#pragma unroll
          for (int k = 0; k < 2; ++k)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb) qf[k][kb] ^= neg;
        }
        const uint64_t rest = bmask & cc.rem;
        start_lookup(rest ? __builtin_ctzll(rest) : -1);
      } else if (lk_phase < 2) {
        lookup_phase();
      }
      barrier_nofence();               // tile i has landed
      if (!busy) continue;
      const int stage = i % kSpStages;
      tile(IntC<0>{}, stage, cc.t, cc.te, first);
      if (two) tile(IntC<1>{}, stage, cc.t, cc.te, first);
      if (last) {
        load_q();                      // the next busy passage's queries
        merge(IntC<0>{});
        if (two) merge(IntC<1>{});
      }
    }
  }
  __syncthreads();

  // O = acc / sum for every row of the chunk; LSE (natural log)
  const size_t obase = (size_t)row0 * H * D + (size_t)h * D;
  for (int e = tid; e < nrows * NC4; e += kSpThreads) {
    const int ri = e / NC4, q = e % NC4;
    const float4 v = reinterpret_cast<const float4*>(Oacc + ri * D)[q ^ (ri & (NC4 - 1))];
    const float l = l_acc[ri];
    const float inv = (l > 0.f) ? 1.f / l : 0.f;
    const size_t off = obase + (size_t)ri * H * D + q * 4;
    if (o_f32) {
      *reinterpret_cast<float4*>(static_cast<float*>(O) + off) =
          make_float4(v.x * inv, v.y * inv, v.z * inv, v.w * inv);
    } else {
      uint2 w;
      w.x = pack2_bf16(v.x * inv, v.y * inv);
      w.y = pack2_bf16(v.z * inv, v.w * inv);
      *reinterpret_cast<uint2*>(static_cast<bf16_t*>(O) + off) = w;
    }
  }
  if (lse && tid < nrows) {
    const float l = l_acc[tid];
    lse[(size_t)(row0 + tid) * H + h] = (l > 0.f) ? (m_acc[tid] + log2f(l)) * kLn2 : -INFINITY;
  }
}

// Standalone work-list launch (calls whose graph is given; the fused route
// builds the list in the edge-selection launch).
constexpr int kPlanThreads = 1024;

__global__ void __launch_bounds__(kPlanThreads)
attn_plan_kernel(const int32_t* __restrict__ kept_offsets,
                 const int32_t* __restrict__ query_passages,
                 const int32_t* __restrict__ passage_offsets, int B, int H, int total_kept,
                 int total_passages, int total_tokens, int k_max, int P_max, int n_ids,
                 int4* __restrict__ items) {
  __shared__ PlanLds L;
  __shared__ uint32_t scan_sh[kPlanThreads / 64 + 1];
  build_attention_plan(L, scan_sh, kept_offsets, query_passages, passage_offsets, B, H,
                       total_kept, total_passages, total_tokens, k_max, P_max, n_ids, items);
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
long long attn_plan_ids(const skip_problem_t& p) {
  if (p.dtype != SKIP_BF16 || p.k_max <= 0 || p.B <= 0 || p.H <= 0) return 0;
  const long long runs = ((long long)p.B * p.H + 7) / 8;
  const long long nch = (p.k_max + kSpRows - 1) / kSpRows;
  return 8 * runs * nch;
}

hipError_t launch_attention_plan(const skip_problem_t& p, const int32_t* kept_offsets,
                                 const int32_t* query_passages,
                                 const int32_t* passage_offsets, int32_t* plan, hipStream_t s) {
  const long long n_ids = attn_plan_ids(p);
  if (n_ids == 0) return hipSuccess;
  if (n_ids > INT32_MAX / 16 || (long long)p.B * p.H > INT32_MAX / 16)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(attn_plan_kernel, dim3(1), dim3(kPlanThreads), 0, s, kept_offsets,
                     query_passages, passage_offsets, p.B, p.H, p.total_kept,
                     p.total_passages, p.total_tokens, p.k_max, p.P_max, (int)n_ids,
                     reinterpret_cast<int4*>(plan));
  return hipGetLastError();
}

hipError_t launch_attention(const skip_problem_t& p, QuerySource q,
                            const int32_t* kept_offsets, const void* Kh, const void* Vh,
                            const int32_t* passage_offsets, const int32_t* query_passages,
                            const uint64_t* rowmask, const int32_t* plan, void* O, float* lse,
                            hipStream_t s) {
  if (p.k_max <= 0) return hipSuccess;
  const int qstride = p.d;
  if (p.dtype == SKIP_BF16) {
    const long long n_ids = attn_plan_ids(p);
    if (n_ids > INT32_MAX / 16 || (long long)p.B * p.H > INT32_MAX / 16)
      return hipErrorInvalidValue;
    const int4* items = reinterpret_cast<const int4*>(plan);
    const float sl2 = p.sm_scale * kLog2e;
#define SKIP_ATTN_SPARSE(DD)                                                                 \
  hipLaunchKernelGGL((attn_sparse_kernel<DD>), dim3((unsigned)n_ids), dim3(kSpThreads),     \
                     0, s, (const bf16_t*)q.base, q.kept_idx, q.N, qstride, (const bf16_t*)Kh, \
                     (const bf16_t*)Vh, passage_offsets, rowmask, items, p.H, p.total_tokens, \
                     sl2, O, p.o_f32, lse)
    if (p.d_h == 64) SKIP_ATTN_SPARSE(64);
    else SKIP_ATTN_SPARSE(128);
#undef SKIP_ATTN_SPARSE
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

// Block-wide exact top-k selection on 64-bit order-preserving keys.
//
// Used for both cuts of the routing core: the kept visual tokens (top k_b
// logits of a question, Def. B.1) and the graph edges (top E_b cosines of a
// question, Def. B.3).  The selected set is: every key above the k-th largest
// key, plus, among keys equal to it, the ones with the lowest element index.
//
// Method: MSB-first radix select with 8-bit digits.  Each pass histograms the
// digits of the keys that still share the chosen prefix, finds the digit at
// which the running count from the top reaches the number still needed, and
// narrows the prefix.  It stops early once every key sharing the prefix is
// needed; after all 8 passes the remaining keys are exactly equal and an
// ordered prefix count admits the lowest indices.  Counts are integers, so
// the result does not depend on thread timing.
//
// Data layout: thread t holds elements [t*C, t*C + cnt) of the n elements in
// registers (keys[0..cnt)), C = ceil(n / blockDim.x) <= MAXPT.
#pragma once

#include <type_traits>

#include "skip_common.h"

namespace skip {

// Two variants of the pass loop share the counting and the final step:
//   * narrow (any block; the prune's 256-thread top-k): histograms alternate
//     between two copies and a pass takes two barriers: wave 0 scans the
//     histogram and broadcasts the digit through LDS.  The next pass's copy
//     is cleared while this one is filled (its last reader, the previous
//     pass's scan, is past a barrier);
//   * wide (1024-thread blocks: the edge selection): histograms rotate over
//     three copies and a pass takes one barrier: every wave scans the
//     histogram itself (no broadcast); the copy the next pass fills is
//     cleared during this pass's counting, when its last readers (the scans
//     two passes back) are past a barrier.  In its first pass most keys share
//     one of a few leading digits (sign and exponent), so a wave counts the
//     keys with its two dominant digits by ballots and adds each count once.
struct SelectShared {
  alignas(16) uint32_t hist[3][256];
  uint32_t misc[2][4];
  uint32_t scan[20];
};

// Inclusive prefix sum over the 64 lanes of a wave: shifts within rows of
// 16 lanes, then the last lane of rows 0 and 2 added to rows 1 and 3, then
// that of row 1 to rows 2 and 3 (DPP row_shr and row_bcast; a lane with no
// source reads 0).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);  // row_shr:8
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);  // row_bcast:15
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return x;
}

// Per-thread element masks: 32 bits, or 64 for more elements a thread.
template <int MAXPT>
using SelectMask = typename std::conditional<(MAXPT > 32), uint64_t, uint32_t>::type;

// Digit of the k-th largest key among those sharing the prefix, from a
// histogram in LDS (digits from the top): lane l holds digits 255 - 4l ..
// 252 - 4l; the first lane whose running count reaches `need` holds it.
// Returns the digit; *above = keys with a larger digit, *inbin = keys with
// this digit.  Wave-uniform results.
__device__ __forceinline__ uint32_t scan_digit(const uint32_t* hist, uint32_t need,
                                               uint32_t* above, uint32_t* inbin) {
  const int lane = threadIdx.x & (kWave - 1);
  const uint4 hv = *reinterpret_cast<const uint4*>(&hist[252 - 4 * lane]);
  const uint32_t h0 = hv.w, h1 = hv.z, h2 = hv.y, h3 = hv.x;   // digits 255-4l, ..
  const uint32_t s = h0 + h1 + h2 + h3;
  const uint32_t inc = wave_incl_scan(s);
  const uint64_t hit = __ballot(inc >= need);
  const int L = hit ? __builtin_ctzll(hit) : kWave - 1;   // (need <= the prefix's count)
  uint32_t c = __builtin_amdgcn_readlane(inc - s, L);
  const uint32_t g0 = __builtin_amdgcn_readlane(h0, L), g1 = __builtin_amdgcn_readlane(h1, L);
  const uint32_t g2 = __builtin_amdgcn_readlane(h2, L), g3 = __builtin_amdgcn_readlane(h3, L);
  uint32_t bin, in;
  if (c + g0 >= need) {
    bin = 255 - 4 * L; in = g0;
  } else if (c + g0 + g1 >= need) {
    c += g0; bin = 254 - 4 * L; in = g1;
  } else if (c + g0 + g1 + g2 >= need) {
    c += g0 + g1; bin = 253 - 4 * L; in = g2;
  } else {
    c += g0 + g1 + g2; bin = 252 - 4 * L; in = g3;
  }
  *above = c;
  *inbin = in;
  return bin;
}

// Returns a bitmask over the thread's elements (bit j = element t*C + j).
// Contains __syncthreads(); a wave may return while others still read the
// last histogram, so a caller that reuses `sh` passes a barrier first.
template <int MAXPT, bool WIDE>
__device__ __forceinline__ SelectMask<MAXPT> block_select_top_impl(
    const uint64_t (&keys)[MAXPT], int cnt, int n, int kk, SelectShared* sh) {
  static_assert(MAXPT <= 64, "flags are at most a 64-bit mask");
  using M = SelectMask<MAXPT>;
  constexpr int W = 8 * sizeof(M);
  constexpr int NH = WIDE ? 3 : 2;                 // histogram copies in rotation
  const M one = 1;
  const M all = (cnt >= W) ? ~(M)0 : ((one << cnt) - one);
  if (kk <= 0) return 0;
  if (kk >= n) return all;
  const int lane = threadIdx.x & (kWave - 1);
  const int C = (n + (int)blockDim.x - 1) / (int)blockDim.x;   // element slots a thread

  for (int i = threadIdx.x; i < 256; i += blockDim.x) sh->hist[0][i] = 0u;
  __syncthreads();
  uint64_t prefix = 0, mask = 0;
  uint32_t need = (uint32_t)kk;
  bool whole_bucket = false;
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
    uint32_t* hist = sh->hist[pass % NH];
    // Count the digits of the keys that share the prefix (element slots up
    // to C = ceil(n / blockDim.x), the same for every thread).
    uint32_t dom0 = 256u, dom1 = 256u, n0 = 0u, n1 = 0u;
    const bool dominant = WIDE && pass == 0;
    if (dominant) {
      const uint32_t dg0 = (uint32_t)(keys[0] >> shift) & 255u;
      const uint64_t a0 = __ballot(0 < cnt);
      if (a0) {
        dom0 = __builtin_amdgcn_readlane(dg0, __builtin_ctzll(a0));
        const uint64_t a1 = __ballot(0 < cnt && dg0 != dom0);
        if (a1) dom1 = __builtin_amdgcn_readlane(dg0, __builtin_ctzll(a1));
      }
    }
#pragma unroll
    for (int j = 0; j < MAXPT; ++j) {
      const bool act = j < cnt && (keys[j] & mask) == prefix;
      const uint32_t dg = (uint32_t)(keys[j] >> shift) & 255u;
      if (j >= C) {
      } else if (dominant) {
        n0 += (uint32_t)__popcll(__ballot(act && dg == dom0));
        n1 += (uint32_t)__popcll(__ballot(act && dg == dom1));
        if (act && dg != dom0 && dg != dom1) atomicAdd(&hist[dg], 1u);
      } else if (act) {
        atomicAdd(&hist[dg], 1u);
      }
    }
    if (dominant && lane == 0) {
      if (n0) atomicAdd(&hist[dom0], n0);
      if (n1) atomicAdd(&hist[dom1], n1);
    }
    for (int i = threadIdx.x; i < 256; i += blockDim.x) sh->hist[(pass + 1) % NH][i] = 0u;
    __syncthreads();
    uint32_t bin, above, inbin;
    if constexpr (WIDE) {
      bin = scan_digit(hist, need, &above, &inbin);
    } else {
      uint32_t* misc = sh->misc[pass & 1];
      if (threadIdx.x < kWave) {
        uint32_t ab, in;
        const uint32_t bn = scan_digit(hist, need, &ab, &in);
        if (lane == 0) {
          misc[0] = bn;
          misc[1] = ab;
          misc[2] = in;
        }
      }
      __syncthreads();
      bin = misc[0];
      above = misc[1];
      inbin = misc[2];
    }
    need -= above;        // candidates with a larger digit: all taken
    prefix |= (uint64_t)bin << shift;
    mask |= 0xffull << shift;
    if (inbin == need) { whole_bucket = true; break; }
  }

  M flags = 0, inb = 0;
#pragma unroll
  for (int j = 0; j < MAXPT; ++j) {
    if (j < cnt) {
      const uint64_t m = keys[j] & mask;
      if (m > prefix) flags |= one << j;
      else if (m == prefix) inb |= one << j;
    }
  }
  if (whole_bucket) return flags | inb;
  // Exactly equal keys: admit the `need` lowest indices.
  uint32_t total;
  uint32_t rank = block_exclusive_scan((uint32_t)__popcll((uint64_t)inb), sh->scan, &total);
#pragma unroll
  for (int j = 0; j < MAXPT; ++j) {
    if (inb & (one << j)) {
      if (rank < need) flags |= one << j;
      ++rank;
    }
  }
  return flags;
}

// Any block size (two barriers a pass).
template <int MAXPT>
__device__ __forceinline__ SelectMask<MAXPT> block_select_top(const uint64_t (&keys)[MAXPT],
                                                              int cnt, int n, int kk,
                                                              SelectShared* sh) {
  return block_select_top_impl<MAXPT, false>(keys, cnt, n, kk, sh);
}

// Blocks of many waves (one barrier a pass, every wave scans).
template <int MAXPT>
__device__ __forceinline__ SelectMask<MAXPT> block_select_top_wide(const uint64_t (&keys)[MAXPT],
                                                                   int cnt, int n, int kk,
                                                                   SelectShared* sh) {
  return block_select_top_impl<MAXPT, true>(keys, cnt, n, kk, sh);
}

}  // namespace skip

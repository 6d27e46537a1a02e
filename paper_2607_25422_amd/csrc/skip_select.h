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

// Histograms and pass results alternate between two copies, so that a pass
// takes two barriers: the next pass's histogram is cleared while this one is
// filled (its last reader, the previous pass's scan, is past a barrier), and
// a pass's result is not overwritten until two passes later.
struct SelectShared {
  uint32_t hist[2][256];
  uint32_t misc[2][4];
  uint32_t scan[20];
};

// Per-thread element masks: 32 bits, or 64 for more elements a thread.
template <int MAXPT>
using SelectMask = typename std::conditional<(MAXPT > 32), uint64_t, uint32_t>::type;

// Returns a bitmask over the thread's elements (bit j = element t*C + j).
template <int MAXPT>
__device__ SelectMask<MAXPT> block_select_top(const uint64_t (&keys)[MAXPT], int cnt, int n,
                                              int kk, SelectShared* sh) {
  static_assert(MAXPT <= 64, "flags are at most a 64-bit mask");
  using M = SelectMask<MAXPT>;
  constexpr int W = 8 * sizeof(M);
  const M one = 1;
  const M all = (cnt >= W) ? ~(M)0 : ((one << cnt) - one);
  if (kk <= 0) return 0;
  if (kk >= n) return all;

  for (int i = threadIdx.x; i < 256; i += blockDim.x) sh->hist[0][i] = 0u;
  __syncthreads();
  uint64_t prefix = 0, mask = 0;
  uint32_t need = (uint32_t)kk;
  bool whole_bucket = false;
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
    uint32_t* hist = sh->hist[pass & 1];
    uint32_t* misc = sh->misc[pass & 1];
#pragma unroll
    for (int j = 0; j < MAXPT; ++j) {
      if (j < cnt && (keys[j] & mask) == prefix)
        atomicAdd(&hist[(uint32_t)(keys[j] >> shift) & 255u], 1u);
    }
    for (int i = threadIdx.x; i < 256; i += blockDim.x) sh->hist[(pass + 1) & 1][i] = 0u;
    __syncthreads();
    if (threadIdx.x < kWave) {
      const int l = threadIdx.x;
      const uint32_t h0 = hist[255 - 4 * l], h1 = hist[254 - 4 * l];
      const uint32_t h2 = hist[253 - 4 * l], h3 = hist[252 - 4 * l];
      const uint32_t s = h0 + h1 + h2 + h3;
      uint32_t inc = s;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        uint32_t y = __shfl_up(inc, o, kWave);
        if (l >= o) inc += y;
      }
      const uint32_t exc = inc - s;
      if (exc < need && need <= inc) {       // exactly one lane
        uint32_t c = exc;
        uint32_t bin, inbin;
        if (c + h0 >= need) {
          bin = 255 - 4 * l; inbin = h0;
        } else if (c + h0 + h1 >= need) {
          c += h0; bin = 254 - 4 * l; inbin = h1;
        } else if (c + h0 + h1 + h2 >= need) {
          c += h0 + h1; bin = 253 - 4 * l; inbin = h2;
        } else {
          c += h0 + h1 + h2; bin = 252 - 4 * l; inbin = h3;
        }
        misc[0] = bin;
        misc[1] = c;        // candidates with a larger digit: all taken
        misc[2] = inbin;    // candidates with exactly this digit
      }
    }
    __syncthreads();
    const uint32_t bin = misc[0], above = misc[1], inbin = misc[2];
    need -= above;
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

}  // namespace skip

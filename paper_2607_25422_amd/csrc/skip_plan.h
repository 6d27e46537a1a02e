// Work list of the passage-major sparse attention (internal to libskip.so),
// built on the device from the offsets by one workgroup of any size.
// Questions are ordered by decreasing cost (chunks x passage tokens, ties to
// the lower index; natural order above kPlanMaxB questions), so that the
// longest items start first.  The (question, head) groups of that order are
// dealt in runs of eight; a run whose groups have at most n chunks takes 8n
// consecutive workgroup ids, chunk c of the run's group i at id base + 8c + i.
// Workgroups are dealt round-robin over the 8 XCDs, so the chunks of one
// (question, head), which read the same K/V tiles, run side by side on one
// XCD and share its L2.  Unused ids get no item (question -1).
//
// Item record (int4): {question, first kept row (global), first passage,
// head | rows << 8 | passages << 16}.
#pragma once

#include "skip_common.h"

namespace skip {

constexpr int kSpRows = 192;              // kept rows per work item
constexpr int kSpMaxP = 64;               // passages per question seen by the attention
constexpr int kPlanMaxB = 2048;           // questions whose order is sorted in LDS

// LDS of the builder: per question the sort key, first kept row, first
// passage, rows, passages and chunks (20 bytes a question).
struct PlanLds {
  uint64_t key[kPlanMaxB];
  int32_t q_k0[kPlanMaxB], q_p0[kPlanMaxB];
  int16_t q_kq[kPlanMaxB];
  uint8_t q_P[kPlanMaxB], q_nch[kPlanMaxB];
};

// The whole block builds the list; scan_sh holds blockDim.x / 64 + 1 words.
// Contains __syncthreads().
__device__ inline void build_attention_plan(PlanLds& L, uint32_t* scan_sh,
                                            const int32_t* __restrict__ kept_offsets,
                                            const int32_t* __restrict__ query_passages,
                                            const int32_t* __restrict__ passage_offsets,
                                            int B, int H, int total_kept, int total_passages,
                                            int total_tokens, int k_max, int P_max, int n_ids,
                                            int4* __restrict__ items) {
  const int tid = threadIdx.x;
  const int nthr = blockDim.x;
  struct Q {
    int k0, kq, p0, P, nch;
  };
  auto question = [&](int b) {
    Q q;
    int k1, p1;
    range_of(kept_offsets, b, total_kept, q.k0, k1);
    range_of(query_passages, b, total_passages, q.p0, p1);
    q.kq = min(k1 - q.k0, k_max);
    q.P = min(min(p1 - q.p0, P_max), kSpMaxP);
    q.nch = (q.kq + kSpRows - 1) / kSpRows;
    return q;
  };
  const bool cached = B <= kPlanMaxB;   // question data and the cost order in LDS
  if (cached) {
    int n = 1;
    while (n < B) n <<= 1;
    for (int b = tid; b < n; b += nthr) {
      uint64_t kk = 0ull;
      if (b < B) {
        const Q q = question(b);
        const int t0 = q.P > 0 ? clampi(passage_offsets[q.p0], 0, total_tokens) : 0;
        const int t1 = q.P > 0 ? clampi(passage_offsets[q.p0 + q.P], t0, total_tokens) : 0;
        const uint64_t cost = (uint64_t)q.nch * (uint64_t)(t1 - t0 + 1);
        kk = (cost << 12) | (uint64_t)(kPlanMaxB - 1 - b);
        L.q_k0[b] = q.k0;
        L.q_p0[b] = q.p0;
        L.q_kq[b] = (int16_t)q.kq;
        L.q_P[b] = (uint8_t)q.P;
        L.q_nch[b] = (uint8_t)q.nch;
      }
      L.key[b] = kk;
    }
    __syncthreads();
    // bitonic sort, descending
    for (int size = 2; size <= n; size <<= 1)
      for (int stride = size >> 1; stride > 0; stride >>= 1) {
        for (int i = tid; i < n; i += nthr) {
          const int jx = i ^ stride;
          if (jx > i) {
            const bool desc = (i & size) == 0;
            const uint64_t x = L.key[i], y = L.key[jx];
            if (desc ? (x < y) : (x > y)) {
              L.key[i] = y;
              L.key[jx] = x;
            }
          }
        }
        __syncthreads();
      }
  }
  // question of rank r, and its data
  auto at = [&](int r, int& b) -> Q {
    if (!cached) {
      b = r;
      return question(r);
    }
    b = kPlanMaxB - 1 - (int)(L.key[r] & (kPlanMaxB - 1));
    return Q{L.q_k0[b], (int)L.q_kq[b], L.q_p0[b], (int)L.q_P[b], (int)L.q_nch[b]};
  };
  const int groups = B * H;   // B * H * k rows fit in int32 (k_max * P_max bounded)
  const int runs = (groups + 7) / 8;
  int carry = 0;
  for (int m0 = 0; m0 < runs; m0 += nthr) {
    const int m = m0 + tid;
    int ncr = 0;
    int qb[8];
    Q qq[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int g = m * 8 + i;
      qb[i] = -1;
      qq[i] = Q{0, 0, 0, 0, 0};
      if (m < runs && g < groups) {
        qq[i] = at(g / H, qb[i]);
        ncr = max(ncr, qq[i].nch);
      }
    }
    uint32_t total;
    const uint32_t pre = block_exclusive_scan((uint32_t)ncr, scan_sh, &total);
    const int base = 8 * (carry + (int)pre);
    if (m < runs)
      for (int c = 0; c < ncr; ++c)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int id = base + 8 * c + i;
          if (id >= n_ids) continue;
          int4 it = make_int4(-1, 0, 0, 0);
          if (qb[i] >= 0 && c < qq[i].nch) {
            const Q& q = qq[i];
            const int rpc = (q.kq + q.nch - 1) / q.nch;
            const int r0 = c * rpc;
            const int nrows = min(q.kq, r0 + rpc) - r0;
            const int h = (m * 8 + i) % H;
            it = make_int4(qb[i], q.k0 + r0, q.p0, h | (nrows << 8) | (q.P << 16));
          }
          items[id] = it;
        }
    carry += (int)total;
  }
  for (int id = 8 * carry + tid; id < n_ids; id += nthr) items[id] = make_int4(-1, 0, 0, 0);
}

}  // namespace skip

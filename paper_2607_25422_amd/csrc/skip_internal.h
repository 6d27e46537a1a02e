// Host-side launchers of the SKIP kernels (internal to libskip.so).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "skip.h"
#include "skip_common.h"

namespace skip {

// Workspace carve-up (byte offsets from the workspace base, 256-B aligned).
struct Workspace {
  double* u;          // [B][d]        scoring vector q_bar/sqrt(d) + w
  double* z;          // [B][N]        salience logits
  double* kbar;       // [total_passages][d] passage keys
  double* part;       // [B][S][k_max][P_max] partial dot products (S slices of d)
  double* qn2;        // [B][S][k_max] partial squared row norms
  double* kn2;        // [B][S][P_max] partial squared passage-key norms
  uint64_t* rowmask;  // [total_kept]  neighbour passages of each kept row
  int32_t* plan;      // [attn_plan_ids][4] attention work list
  int32_t* counters;  // [B] scoring workgroups finished per question
  size_t bytes;
};

Workspace carve_workspace(const skip_problem_t& p, void* base);

// Stage 1 ---------------------------------------------------------------
hipError_t launch_pool_question(const skip_problem_t& p, const void* Qtok,
                                const int32_t* q_offsets, const void* w_bias,
                                double* u, int32_t* counters, hipStream_t s);
// Scoring and top-k of every question in one launch (u and the cleared
// counters from launch_pool_question), plus the pooling of n_keys passage
// keys of Kh into kbar (0: none).
hipError_t launch_prune(const skip_problem_t& p, const void* V, const double* u, double* z,
                        float* scores, const int32_t* kept_offsets, int32_t* kept_idx,
                        int32_t* counters, const void* Kh, const int32_t* passage_offsets,
                        int n_keys, double* kbar, hipStream_t s);
hipError_t launch_topk(const skip_problem_t& p, const double* z,
                       const int32_t* kept_offsets, int32_t* kept_idx,
                       hipStream_t s);
hipError_t launch_gather(const skip_problem_t& p, const void* V,
                         const int32_t* kept_offsets, const int32_t* kept_idx,
                         void* V_kept, hipStream_t s);

// Main-text scorer (two-layer perceptron) -------------------------------
struct MlpScratch {
  bf16_t* qbf;       // [B][d]         q_bar rounded to bf16
  float* cvec;       // [B][h]         W1[:, d:2d] q_bar' + b1
  float* sp;         // [h/128][B][N]  partial scores per 128 hidden units
  u32x4* wpack;      // [h][2d] bf16   W1's v and Hadamard blocks in fragment order
};
size_t mlp_scratch_bytes(const skip_problem_t& p, int hidden);
MlpScratch carve_mlp_scratch(const skip_problem_t& p, int hidden, void* base);
hipError_t launch_mlp_scores(const skip_problem_t& p, const skip_qvs_mlp_t& m, const void* V,
                             const double* qbar, MlpScratch ms, double* z, float* scores,
                             hipStream_t s);

// Passage verification gate ---------------------------------------------
struct GateScratch {
  double* qbar;      // [B][d]         mean of the question tokens
  double* vbar;      // [B][d]         mean of the kept visual rows
  bf16_t* X;         // [T][3d]        passage blocks of the gate inputs
  bf16_t* Xq;        // [B][2d]        question blocks of the gate inputs
  float* part;       // [S][T][h]      chunk partials of the passage blocks' products
  float* partq;      // [Sq][B][h]     chunk partials of the question blocks' products
  float* z;          // [T]            logits
  int32_t* pq;       // [T]            question of each passage
  int32_t* done;     // [B]            finished passages per question
};
size_t gate_scratch_bytes(const skip_problem_t& p, int hidden);
GateScratch carve_gate_scratch(const skip_problem_t& p, int hidden, void* base);
// g.qbar, g.vbar from the question tokens and the kept rows (rows[kept
// range] when kept_idx is NULL, else V[b][kept_idx[r]], rows = V), and the
// gate inputs g.X, g.Xq from them and the passage keys (kbar, or
// passage_keys if given; complete before this launch)
hipError_t launch_gate_means(const skip_problem_t& p, const void* Qtok,
                             const int32_t* q_offsets, const void* rows,
                             const int32_t* kept_offsets, const int32_t* kept_idx,
                             const double* kbar, const float* passage_keys,
                             const int32_t* query_passages, GateScratch g, hipStream_t s);
// the gate on the inputs launch_gate_means wrote
hipError_t launch_gate(const skip_problem_t& p, const skip_skv_gate_t& gt,
                       const int32_t* query_passages, GateScratch g, float* logits,
                       uint8_t* keep, hipStream_t s);

// Learned projection of the kept rows --------------------------------------
size_t proj_scratch_bytes(int d, int d_out);
hipError_t launch_proj_pack(int d, int d_out, const void* W, void* packed, hipStream_t s);
hipError_t launch_proj_gemm(const skip_problem_t& p, const void* rows, const int32_t* kept_offsets,
                            const int32_t* kept_idx, const void* packed, int d_out, void* Y,
                            int out_f32, hipStream_t s);
hipError_t launch_keys_bf16(const double* kbar, const float* given, size_t n, void* out,
                            hipStream_t s);
hipError_t launch_project(const skip_problem_t& p, const void* rows, const int32_t* kept_offsets,
                          const int32_t* kept_idx, const void* W, int d_out, void* Y,
                          int out_f32, void* scratch, hipStream_t s);

// Regions of the kept tokens (k-means) ------------------------------------
int region_slices(const skip_problem_t& p);
size_t region_scratch_bytes(const skip_problem_t& p, int r_max);
// rows: the kept rows (kept_idx NULL) or V read through kept_idx
hipError_t launch_regions(const skip_problem_t& p, const void* rows, const int32_t* kept_offsets,
                          const int32_t* kept_idx, int r_max, int n_iter, int32_t* region,
                          float* centroids, int32_t* sizes, void* scratch, hipStream_t s);

// Stage 2 ---------------------------------------------------------------
// Query rows: if kept_idx is non-NULL, row r of question b is
// V[b][kept_idx[r]] (the fused route); otherwise it is Qh[r].
struct QuerySource {
  const void* base;
  const int32_t* kept_idx;   // NULL for Qh
  int32_t N;                 // visual tokens per question (fused route)
};

hipError_t launch_passage_keys(const skip_problem_t& p, const void* Kh,
                               const int32_t* passage_offsets, double* kbar,
                               hipStream_t s);
struct EdgePartials {
  double* part;              // per-slice partial dot products
  double* qn2;               // per-slice partial squared row norms
  double* kn2;               // per-slice partial squared passage-key norms
};
int edge_slices(const skip_problem_t& p);
hipError_t launch_edge_dot(const skip_problem_t& p, QuerySource q,
                           const int32_t* kept_offsets,
                           const int32_t* query_passages, const double* kbar,
                           const float* passage_keys, EdgePartials ep, hipStream_t s);
hipError_t launch_edge_select(const skip_problem_t& p, EdgePartials ep,
                              const int32_t* kept_offsets, const int32_t* query_passages,
                              uint64_t* rowmask, int32_t* rowptr_out, int32_t* col_out,
                              hipStream_t s, const uint8_t* passage_keep = nullptr,
                              const int32_t* passage_offsets = nullptr,
                              int32_t* plan = nullptr);
hipError_t launch_csr_to_mask(const skip_problem_t& p, const int32_t* kept_offsets,
                              const int32_t* query_passages,
                              const int32_t* edge_rowptr, const int32_t* edge_col,
                              uint64_t* rowmask, hipStream_t s);
// Workgroup ids of the bf16 attention launch (0 for fp32): the work list
// takes one 16-byte record per id.
long long attn_plan_ids(const skip_problem_t& p);
// Work list of the bf16 attention launch (depends on the offsets only).
hipError_t launch_attention_plan(const skip_problem_t& p, const int32_t* kept_offsets,
                                 const int32_t* query_passages,
                                 const int32_t* passage_offsets, int32_t* plan, hipStream_t s);
hipError_t launch_attention(const skip_problem_t& p, QuerySource q,
                            const int32_t* kept_offsets, const void* Kh,
                            const void* Vh, const int32_t* passage_offsets,
                            const int32_t* query_passages,
                            const uint64_t* rowmask, const int32_t* plan, void* O, float* lse,
                            hipStream_t s);

}  // namespace skip

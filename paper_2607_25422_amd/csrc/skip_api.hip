// C ABI of libskip.so: argument validation, workspace carving, launches.
// The public contract (argument meaning, layout, ownership, errors) is in
// include/skip.h.
#include <cmath>
#include <cstdint>
#include <mutex>

#include "skip.h"
#include "skip_internal.h"
#include "skip_pool.h"

namespace skip {
namespace {

constexpr size_t kAlign = 256;
constexpr int kMaxN = 16384;
constexpr int kMaxD = 8192;
constexpr int kMaxCandidates = 16384;   // k_b * P_b per question

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

enum Need { kPrune = 1, kGraph = 2 };

skip_status_t check_common(const skip_problem_t* p) {
  if (!p) return SKIP_ERR_INVALID_ARG;
  if (p->o_f32 != 0 && p->o_f32 != 1) return SKIP_ERR_INVALID_ARG;
  if (p->dtype != SKIP_F32 && p->dtype != SKIP_BF16) return SKIP_ERR_INVALID_ARG;
  if (p->B < 1 || p->d < 1 || p->k_max < 0 || p->total_kept < 0) return SKIP_ERR_INVALID_ARG;
  if ((int64_t)p->total_kept > (int64_t)p->B * p->k_max) return SKIP_ERR_INVALID_ARG;
  if (p->total_kept < p->k_max) return SKIP_ERR_INVALID_ARG;
  if (p->d % 8 != 0 || p->d > kMaxD) return SKIP_ERR_UNSUPPORTED;
  return SKIP_OK;
}

// Element arrays are read with 16-byte vector and direct-to-LDS loads: a
// misaligned array is an argument error (NULL passes; required pointers are
// checked separately).
static bool al16(const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15) == 0; }

static_assert(sizeof(skip_problem_t) == 88 && offsetof(skip_problem_t, avg_degree) == 56 &&
                  offsetof(skip_problem_t, edge_rule) == 72 &&
                  offsetof(skip_problem_t, edge_beta) == 80,
              "skip_problem_t layout is part of the ABI");

skip_status_t check(const skip_problem_t* p, int need) {
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (need & kPrune) {
    if (p->N < 1 || p->total_qtok < p->B) return SKIP_ERR_INVALID_ARG;
    if (p->k_max > p->N) return SKIP_ERR_INVALID_ARG;
    if (p->N > kMaxN) return SKIP_ERR_UNSUPPORTED;
    if ((int64_t)p->B * p->N > INT32_MAX) return SKIP_ERR_UNSUPPORTED;
  }
  if (need & kGraph) {
    if (p->H < 1 || p->d_h < 1 || (int64_t)p->H * p->d_h != p->d) return SKIP_ERR_INVALID_ARG;
    if (p->d_h != 64 && p->d_h != 128) return SKIP_ERR_UNSUPPORTED;
    if (p->P_max < 0 || p->total_passages < p->P_max) return SKIP_ERR_INVALID_ARG;
    if ((int64_t)p->total_passages > (int64_t)p->B * p->P_max) return SKIP_ERR_INVALID_ARG;
    if (p->total_tokens < p->total_passages) return SKIP_ERR_INVALID_ARG;
    if (p->total_passages > 0 && (p->L_max < 1 || p->L_max > p->total_tokens))
      return SKIP_ERR_INVALID_ARG;
    if (!std::isfinite(p->avg_degree) || p->avg_degree < 0.0) return SKIP_ERR_INVALID_ARG;
    if (p->edge_rule != SKIP_EDGE_QUESTION_BUDGET && p->edge_rule != SKIP_EDGE_ROW_TOP &&
        p->edge_rule != SKIP_EDGE_TOP_FRACTION)
      return SKIP_ERR_INVALID_ARG;
    if (p->edge_metric != SKIP_EDGE_COSINE && p->edge_metric != SKIP_EDGE_DOT)
      return SKIP_ERR_INVALID_ARG;
    if (p->edge_rule == SKIP_EDGE_TOP_FRACTION &&
        !(p->edge_beta > 0.0 && p->edge_beta <= 1.0))
      return SKIP_ERR_INVALID_ARG;
    if (!std::isfinite(p->sm_scale)) return SKIP_ERR_INVALID_ARG;
    if (p->total_edges < 0) return SKIP_ERR_INVALID_ARG;
    if (p->P_max > 64) return SKIP_ERR_UNSUPPORTED;
    if ((int64_t)p->k_max * p->P_max > kMaxCandidates) return SKIP_ERR_UNSUPPORTED;
  }
  return SKIP_OK;
}

size_t workspace_size(const skip_problem_t& p) {
  size_t n = 0;
  n += align_up((size_t)p.B * p.d * sizeof(double));                  // u
  n += align_up((size_t)p.B * (size_t)p.N * sizeof(double));          // z
  n += align_up((size_t)p.total_passages * p.d * sizeof(double));     // kbar
  const size_t S = (size_t)edge_slices(p);
  n += align_up((size_t)p.B * S * p.k_max * p.P_max * sizeof(double));  // edge partials
  n += align_up((size_t)p.B * S * p.k_max * sizeof(double));            // row norms
  n += align_up((size_t)p.B * S * p.P_max * sizeof(double));            // key norms
  n += align_up((size_t)p.total_kept * sizeof(uint64_t));             // rowmask
  n += align_up((size_t)attn_plan_ids(p) * 4 * sizeof(int32_t));      // attention work list
  n += align_up((size_t)p.B * sizeof(int32_t));                       // prune counters
  return n;
}

#define SKIP_TRY(expr)                       \
  do {                                       \
    hipError_t e_ = (expr);                  \
    if (e_ != hipSuccess) return SKIP_ERR_HIP; \
  } while (0)

}  // namespace

Workspace carve_workspace(const skip_problem_t& p, void* base) {
  Workspace w{};
  char* c = static_cast<char*>(base);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* r = c + off;
    off += align_up(bytes);
    return r;
  };
  w.u = reinterpret_cast<double*>(take((size_t)p.B * p.d * sizeof(double)));
  w.z = reinterpret_cast<double*>(take((size_t)p.B * (size_t)p.N * sizeof(double)));
  w.kbar = reinterpret_cast<double*>(take((size_t)p.total_passages * p.d * sizeof(double)));
  const size_t S = (size_t)edge_slices(p);
  w.part = reinterpret_cast<double*>(take((size_t)p.B * S * p.k_max * p.P_max * sizeof(double)));
  w.qn2 = reinterpret_cast<double*>(take((size_t)p.B * S * p.k_max * sizeof(double)));
  w.kn2 = reinterpret_cast<double*>(take((size_t)p.B * S * p.P_max * sizeof(double)));
  w.rowmask = reinterpret_cast<uint64_t*>(take((size_t)p.total_kept * sizeof(uint64_t)));
  w.plan = reinterpret_cast<int32_t*>(take((size_t)attn_plan_ids(p) * 4 * sizeof(int32_t)));
  w.counters = reinterpret_cast<int32_t*>(take((size_t)p.B * sizeof(int32_t)));
  w.bytes = off;
  return w;
}

}  // namespace skip

using namespace skip;

extern "C" {

int32_t skip_abi_version(void) { return SKIP_ABI_VERSION; }

const char* skip_status_string(skip_status_t s) {
  switch (s) {
    case SKIP_OK: return "SKIP_OK";
    case SKIP_ERR_INVALID_ARG: return "SKIP_ERR_INVALID_ARG: invalid argument";
    case SKIP_ERR_UNSUPPORTED: return "SKIP_ERR_UNSUPPORTED: shape not implemented";
    case SKIP_ERR_WORKSPACE: return "SKIP_ERR_WORKSPACE: workspace too small";
    case SKIP_ERR_HIP: return "SKIP_ERR_HIP: HIP launch failed";
  }
  return "SKIP_ERR_UNKNOWN";
}

skip_status_t skip_workspace_bytes(const skip_problem_t* p, size_t* bytes) {
  if (!bytes) return SKIP_ERR_INVALID_ARG;
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (p->N < 0 || p->P_max < 0 || p->total_passages < 0) return SKIP_ERR_INVALID_ARG;
  *bytes = workspace_size(*p);
  return SKIP_OK;
}

skip_status_t skip_prune_topk(const skip_problem_t* p, const void* V, const void* Qtok,
                              const int32_t* q_offsets, const void* w_bias,
                              const int32_t* kept_offsets, int32_t* kept_idx, float* scores,
                              void* V_kept, void* workspace, size_t workspace_bytes,
                              void* stream) {
  skip_status_t st = check(p, kPrune);
  if (st != SKIP_OK) return st;
  if (!V || !Qtok || !q_offsets || !kept_offsets || !workspace) return SKIP_ERR_INVALID_ARG;
  if (p->total_kept > 0 && !kept_idx) return SKIP_ERR_INVALID_ARG;
  if (!al16(V) || !al16(Qtok) || !al16(w_bias) || !al16(V_kept)) return SKIP_ERR_INVALID_ARG;
  if (workspace_bytes < workspace_size(*p)) return SKIP_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Workspace w = carve_workspace(*p, workspace);
  SKIP_TRY(launch_pool_question(*p, Qtok, q_offsets, w_bias, w.u, w.counters, s));
  SKIP_TRY(launch_prune(*p, V, w.u, w.z, scores, kept_offsets, kept_idx, w.counters, nullptr,
                        nullptr, 0, nullptr, s));
  if (p->total_kept > 0 && V_kept)
    SKIP_TRY(launch_gather(*p, V, kept_offsets, kept_idx, V_kept, s));
  return SKIP_OK;
}

static_assert(sizeof(skip_qvs_mlp_t) == 40 && offsetof(skip_qvs_mlp_t, b2) == 32,
              "skip_qvs_mlp_t layout is part of the ABI");

static bool mlp_shape_ok(const skip_qvs_mlp_t* m) {
  return m->hidden > 0 && m->hidden % 256 == 0 && m->hidden <= 4096;
}

skip_status_t skip_workspace_bytes_mlp(const skip_problem_t* p, int32_t hidden, size_t* bytes) {
  if (!bytes) return SKIP_ERR_INVALID_ARG;
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (p->N < 0 || p->P_max < 0 || p->total_passages < 0) return SKIP_ERR_INVALID_ARG;
  if (hidden <= 0) return SKIP_ERR_INVALID_ARG;
  if (hidden % 256 != 0 || hidden > 4096) return SKIP_ERR_UNSUPPORTED;
  *bytes = workspace_size(*p) + mlp_scratch_bytes(*p, hidden);
  return SKIP_OK;
}

skip_status_t skip_prune_topk_mlp(const skip_problem_t* p, const skip_qvs_mlp_t* mlp,
                                  const void* V, const void* Qtok, const int32_t* q_offsets,
                                  const int32_t* kept_offsets, int32_t* kept_idx,
                                  float* scores, void* V_kept, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  skip_status_t st = check(p, kPrune);
  if (st != SKIP_OK) return st;
  if (!mlp || !V || !Qtok || !q_offsets || !kept_offsets || !workspace)
    return SKIP_ERR_INVALID_ARG;
  if (p->total_kept > 0 && !kept_idx) return SKIP_ERR_INVALID_ARG;
  if (mlp->reserved != 0 || !mlp->W1 || !mlp->w2 || mlp->hidden <= 0 ||
      !std::isfinite(mlp->b2))
    return SKIP_ERR_INVALID_ARG;
  if (!al16(V) || !al16(Qtok) || !al16(V_kept) || !al16(mlp->W1)) return SKIP_ERR_INVALID_ARG;
  if (p->dtype != SKIP_BF16 || p->d % 32 != 0 || !mlp_shape_ok(mlp)) return SKIP_ERR_UNSUPPORTED;
  if ((int64_t)mlp->hidden * 3 * p->d > INT32_MAX) return SKIP_ERR_UNSUPPORTED;
  const size_t need = workspace_size(*p) + mlp_scratch_bytes(*p, mlp->hidden);
  if (workspace_bytes < need) return SKIP_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Workspace w = carve_workspace(*p, workspace);
  MlpScratch ms = carve_mlp_scratch(*p, mlp->hidden, static_cast<char*>(workspace) + w.bytes);
  // q_bar itself (the plain mean of the question tokens) into u
  SKIP_TRY(launch_pools(p->dtype, p->d, nullptr, nullptr, 0, 0, nullptr, nullptr, Qtok,
                        q_offsets, p->B, p->total_qtok, w.u, s));
  SKIP_TRY(launch_mlp_scores(*p, *mlp, V, w.u, ms, w.z, scores, s));
  if (p->total_kept > 0) {
    SKIP_TRY(launch_topk(*p, w.z, kept_offsets, kept_idx, s));
    if (V_kept) SKIP_TRY(launch_gather(*p, V, kept_offsets, kept_idx, V_kept, s));
  }
  return SKIP_OK;
}

static skip_status_t xattn_impl(const skip_problem_t* p, const void* Qh, const void* edge_rows,
                                const int32_t* kept_offsets, const void* Kh, const void* Vh,
                                const int32_t* passage_offsets, const int32_t* query_passages,
                                const float* passage_keys, const int32_t* edge_rowptr,
                                const int32_t* edge_col, const uint8_t* passage_keep, void* O,
                                float* lse, int32_t* edge_rowptr_out, int32_t* edge_col_out,
                                void* workspace, size_t workspace_bytes, void* stream) {
  skip_status_t st = check(p, kGraph);
  if (st != SKIP_OK) return st;
  if (!kept_offsets || !query_passages || !passage_offsets || !workspace)
    return SKIP_ERR_INVALID_ARG;
  if (p->total_kept > 0 && (!Qh || !O)) return SKIP_ERR_INVALID_ARG;
  if (p->total_tokens > 0 && (!Kh || !Vh)) return SKIP_ERR_INVALID_ARG;
  if (!al16(Qh) || !al16(edge_rows) || !al16(Kh) || !al16(Vh) || !al16(O) ||
      !al16(passage_keys))
    return SKIP_ERR_INVALID_ARG;
  const bool given = edge_rowptr || edge_col;
  if (given && (!edge_rowptr || (!edge_col && p->total_edges > 0))) return SKIP_ERR_INVALID_ARG;
  if ((edge_rowptr_out == nullptr) != (edge_col_out == nullptr)) return SKIP_ERR_INVALID_ARG;
  if (given && edge_rowptr_out) return SKIP_ERR_INVALID_ARG;
  if (workspace_bytes < workspace_size(*p)) return SKIP_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Workspace w = carve_workspace(*p, workspace);
  const EdgePartials ep{w.part, w.qn2, w.kn2};
  if (p->total_kept == 0) {
    // No kept rows: only the (empty) CSR needs its closing offset.
    if (edge_rowptr_out)
      SKIP_TRY(launch_edge_select(*p, ep, kept_offsets, query_passages, w.rowmask,
                                  edge_rowptr_out, edge_col_out, s, passage_keep));
    return SKIP_OK;
  }
  QuerySource q{Qh, nullptr, 0};
  if (given) {
    SKIP_TRY(launch_csr_to_mask(*p, kept_offsets, query_passages, edge_rowptr, edge_col,
                                w.rowmask, s));
  } else {
    if (!passage_keys) SKIP_TRY(launch_passage_keys(*p, Kh, passage_offsets, w.kbar, s));
    const QuerySource e{edge_rows ? edge_rows : Qh, nullptr, 0};
    SKIP_TRY(launch_edge_dot(*p, e, kept_offsets, query_passages, w.kbar, passage_keys, ep, s));
    // the selection launch also builds the attention's work list
    SKIP_TRY(launch_edge_select(*p, ep, kept_offsets, query_passages, w.rowmask,
                                edge_rowptr_out, edge_col_out, s, passage_keep,
                                passage_offsets, w.plan));
  }
  if (given)
    SKIP_TRY(launch_attention_plan(*p, kept_offsets, query_passages, passage_offsets, w.plan, s));
  SKIP_TRY(launch_attention(*p, q, kept_offsets, Kh, Vh, passage_offsets, query_passages,
                            w.rowmask, w.plan, O, lse, s));
  return SKIP_OK;
}

skip_status_t skip_bipartite_xattn(const skip_problem_t* p, const void* Qh,
                                   const int32_t* kept_offsets, const void* Kh, const void* Vh,
                                   const int32_t* passage_offsets,
                                   const int32_t* query_passages, const float* passage_keys,
                                   const int32_t* edge_rowptr, const int32_t* edge_col,
                                   void* O, float* lse, int32_t* edge_rowptr_out,
                                   int32_t* edge_col_out, void* workspace,
                                   size_t workspace_bytes, void* stream) {
  return xattn_impl(p, Qh, nullptr, kept_offsets, Kh, Vh, passage_offsets, query_passages,
                    passage_keys, edge_rowptr, edge_col, nullptr, O, lse, edge_rowptr_out,
                    edge_col_out, workspace, workspace_bytes, stream);
}

skip_status_t skip_bipartite_xattn_masked(const skip_problem_t* p, const void* Qh,
                                          const int32_t* kept_offsets, const void* Kh,
                                          const void* Vh, const int32_t* passage_offsets,
                                          const int32_t* query_passages,
                                          const float* passage_keys,
                                          const uint8_t* passage_keep, void* O, float* lse,
                                          int32_t* edge_rowptr_out, int32_t* edge_col_out,
                                          void* workspace, size_t workspace_bytes,
                                          void* stream) {
  if (!passage_keep && p && p->total_passages > 0) return SKIP_ERR_INVALID_ARG;
  return xattn_impl(p, Qh, nullptr, kept_offsets, Kh, Vh, passage_offsets, query_passages,
                    passage_keys, nullptr, nullptr, passage_keep, O, lse, edge_rowptr_out,
                    edge_col_out, workspace, workspace_bytes, stream);
}

skip_status_t skip_bipartite_xattn_proj(const skip_problem_t* p, const void* Qh,
                                        const void* edge_rows, const int32_t* kept_offsets,
                                        const void* Kh, const void* Vh,
                                        const int32_t* passage_offsets,
                                        const int32_t* query_passages,
                                        const float* passage_keys,
                                        const uint8_t* passage_keep, void* O, float* lse,
                                        int32_t* edge_rowptr_out, int32_t* edge_col_out,
                                        void* workspace, size_t workspace_bytes,
                                        void* stream) {
  if (!p) return SKIP_ERR_INVALID_ARG;
  if (p->total_kept > 0 && !edge_rows) return SKIP_ERR_INVALID_ARG;
  if (p->total_passages > 0 && !passage_keys) return SKIP_ERR_INVALID_ARG;
  return xattn_impl(p, Qh, edge_rows, kept_offsets, Kh, Vh, passage_offsets, query_passages,
                    passage_keys, nullptr, nullptr, passage_keep, O, lse, edge_rowptr_out,
                    edge_col_out, workspace, workspace_bytes, stream);
}

skip_status_t skip_workspace_bytes_project(const skip_problem_t* p, int32_t d_out,
                                           size_t* bytes) {
  if (!bytes) return SKIP_ERR_INVALID_ARG;
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (d_out <= 0) return SKIP_ERR_INVALID_ARG;
  if (d_out % 256 != 0 || d_out > 65536) return SKIP_ERR_UNSUPPORTED;
  *bytes = proj_scratch_bytes(p->d, d_out);
  return SKIP_OK;
}

// Shared argument checks of the projection calls (W: the weights, or their
// packed copy).
static skip_status_t check_project(const skip_problem_t* p, const void* rows,
                                   const int32_t* kept_offsets, const int32_t* kept_idx,
                                   const void* W, int32_t d_out, const void* Y,
                                   int32_t out_f32) {
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (!W || (out_f32 != 0 && out_f32 != 1) || d_out <= 0) return SKIP_ERR_INVALID_ARG;
  if (p->total_kept > 0 && (!rows || !Y)) return SKIP_ERR_INVALID_ARG;
  if (kept_idx && !kept_offsets) return SKIP_ERR_INVALID_ARG;
  if (!al16(W) || !al16(rows) || !al16(Y)) return SKIP_ERR_INVALID_ARG;
  if (p->dtype != SKIP_BF16 || p->d % 32 != 0 || d_out % 256 != 0 || d_out > 65536)
    return SKIP_ERR_UNSUPPORTED;
  if (kept_idx) {
    if (p->N < 1 || p->k_max > p->N) return SKIP_ERR_INVALID_ARG;
    if ((int64_t)p->B * p->N > INT32_MAX) return SKIP_ERR_UNSUPPORTED;
  }
  return SKIP_OK;
}

skip_status_t skip_gather_project(const skip_problem_t* p, const void* rows,
                                  const int32_t* kept_offsets, const int32_t* kept_idx,
                                  const void* W, int32_t d_out, void* Y, int32_t out_f32,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  skip_status_t st = check_project(p, rows, kept_offsets, kept_idx, W, d_out, Y, out_f32);
  if (st != SKIP_OK) return st;
  if (!workspace || !al16(workspace)) return SKIP_ERR_INVALID_ARG;
  if (workspace_bytes < proj_scratch_bytes(p->d, d_out)) return SKIP_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  SKIP_TRY(launch_project(*p, rows, kept_offsets, kept_idx, W, d_out, Y, out_f32, workspace, s));
  return SKIP_OK;
}

skip_status_t skip_pack_projection(const skip_problem_t* p, const void* W, int32_t d_out,
                                   void* packed, size_t packed_bytes, void* stream) {
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (!W || !packed || d_out <= 0 || !al16(W) || !al16(packed)) return SKIP_ERR_INVALID_ARG;
  if (p->dtype != SKIP_BF16 || p->d % 32 != 0 || d_out % 256 != 0 || d_out > 65536)
    return SKIP_ERR_UNSUPPORTED;
  if (packed_bytes < proj_scratch_bytes(p->d, d_out)) return SKIP_ERR_WORKSPACE;
  SKIP_TRY(launch_proj_pack(p->d, d_out, W, packed, static_cast<hipStream_t>(stream)));
  return SKIP_OK;
}

skip_status_t skip_gather_project_packed(const skip_problem_t* p, const void* rows,
                                         const int32_t* kept_offsets, const int32_t* kept_idx,
                                         const void* packed, int32_t d_out, void* Y,
                                         int32_t out_f32, void* stream) {
  skip_status_t st = check_project(p, rows, kept_offsets, kept_idx, packed, d_out, Y, out_f32);
  if (st != SKIP_OK) return st;
  SKIP_TRY(launch_proj_gemm(*p, rows, kept_offsets, kept_idx, packed, d_out, Y, out_f32,
                            static_cast<hipStream_t>(stream)));
  return SKIP_OK;
}

// Workspace of skip_project_passage_keys: pooled keys (double), the keys as
// bf16 rows, W repacked.
static size_t project_keys_bytes(const skip_problem_t& p, int32_t d_out) {
  const size_t n = (size_t)p.total_passages * p.d;
  return align_up(n * sizeof(double)) + align_up(n * sizeof(bf16_t)) +
         proj_scratch_bytes(p.d, d_out);
}

skip_status_t skip_workspace_bytes_project_keys(const skip_problem_t* p, int32_t d_out,
                                                size_t* bytes) {
  if (!bytes) return SKIP_ERR_INVALID_ARG;
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (d_out <= 0) return SKIP_ERR_INVALID_ARG;
  if (d_out % 256 != 0 || d_out > 65536) return SKIP_ERR_UNSUPPORTED;
  *bytes = project_keys_bytes(*p, d_out);
  return SKIP_OK;
}

skip_status_t skip_project_passage_keys(const skip_problem_t* p, const void* Kh,
                                        const int32_t* passage_offsets,
                                        const float* passage_keys, const void* W,
                                        int32_t d_out, float* keys_out, void* workspace,
                                        size_t workspace_bytes, void* stream) {
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (!W || d_out <= 0 || !al16(W)) return SKIP_ERR_INVALID_ARG;
  if (p->dtype != SKIP_BF16 || p->d % 32 != 0 || d_out % 256 != 0 || d_out > 65536)
    return SKIP_ERR_UNSUPPORTED;
  if (p->total_passages > 0) {
    if (!keys_out || !al16(keys_out)) return SKIP_ERR_INVALID_ARG;
    if (passage_keys ? !al16(passage_keys) : (!Kh || !passage_offsets || !al16(Kh)))
      return SKIP_ERR_INVALID_ARG;
  }
  if (!workspace || !al16(workspace)) return SKIP_ERR_INVALID_ARG;
  if (workspace_bytes < project_keys_bytes(*p, d_out)) return SKIP_ERR_WORKSPACE;
  if (p->total_passages == 0) return SKIP_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const size_t n = (size_t)p->total_passages * p->d;
  char* ws = static_cast<char*>(workspace);
  double* kbar = reinterpret_cast<double*>(ws);
  void* kb = ws + align_up(n * sizeof(double));
  void* packed = static_cast<char*>(kb) + align_up(n * sizeof(bf16_t));
  if (!passage_keys) SKIP_TRY(launch_passage_keys(*p, Kh, passage_offsets, kbar, s));
  SKIP_TRY(launch_keys_bf16(kbar, passage_keys, n, kb, s));
  // the keys are the rows of a plain (ungathered) projection
  skip_problem_t q = *p;
  q.total_kept = p->total_passages;
  SKIP_TRY(launch_project(q, kb, nullptr, nullptr, W, d_out, keys_out, 1, packed, s));
  return SKIP_OK;
}

static_assert(sizeof(skip_skv_gate_t) == 56 && offsetof(skip_skv_gate_t, b2) == 32 &&
                  offsetof(skip_skv_gate_t, rho) == 48,
              "skip_skv_gate_t layout is part of the ABI");

static bool gate_hidden_ok(int32_t hidden) {
  return hidden % 64 == 0 && hidden <= 4096;
}

// gate fields and the shapes the gate kernels take (p already checked)
static skip_status_t check_gate(const skip_problem_t* p, const skip_skv_gate_t* gate) {
  if (gate->reserved != 0 || !gate->W || !gate->w2 || gate->hidden <= 0 ||
      !std::isfinite(gate->b2) || !(gate->tau > 0.0 && gate->tau < 1.0) ||
      !(gate->rho > 0.0 && gate->rho <= 1.0))
    return SKIP_ERR_INVALID_ARG;
  if (reinterpret_cast<uintptr_t>(gate->W) % 16 != 0) return SKIP_ERR_INVALID_ARG;
  if (p->dtype != SKIP_BF16 || p->d % 32 != 0 || !gate_hidden_ok(gate->hidden))
    return SKIP_ERR_UNSUPPORTED;
  if ((int64_t)gate->hidden * 5 * p->d > INT32_MAX) return SKIP_ERR_UNSUPPORTED;
  return SKIP_OK;
}

skip_status_t skip_workspace_bytes_gate(const skip_problem_t* p, int32_t hidden, size_t* bytes) {
  if (!bytes) return SKIP_ERR_INVALID_ARG;
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (p->N < 0 || p->P_max < 0 || p->total_passages < 0) return SKIP_ERR_INVALID_ARG;
  if (hidden <= 0) return SKIP_ERR_INVALID_ARG;
  if (!gate_hidden_ok(hidden)) return SKIP_ERR_UNSUPPORTED;
  *bytes = workspace_size(*p) + gate_scratch_bytes(*p, hidden);
  return SKIP_OK;
}

skip_status_t skip_skv_gate(const skip_problem_t* p, const skip_skv_gate_t* gate,
                            const void* Qtok, const int32_t* q_offsets, const void* V_kept,
                            const int32_t* kept_offsets, const void* Kh,
                            const int32_t* passage_offsets, const int32_t* query_passages,
                            const float* passage_keys, float* logits, uint8_t* keep,
                            void* workspace, size_t workspace_bytes, void* stream) {
  skip_status_t st = check(p, kGraph);
  if (st != SKIP_OK) return st;
  if (!gate || !Qtok || !q_offsets || !kept_offsets || !query_passages || !workspace)
    return SKIP_ERR_INVALID_ARG;
  if (p->total_qtok < p->B) return SKIP_ERR_INVALID_ARG;
  if (p->total_kept > 0 && !V_kept) return SKIP_ERR_INVALID_ARG;
  if (p->total_passages > 0 && !keep) return SKIP_ERR_INVALID_ARG;
  if (!al16(Qtok) || !al16(V_kept) || !al16(Kh) || !al16(passage_keys))
    return SKIP_ERR_INVALID_ARG;
  if (!passage_keys && p->total_passages > 0 && (!Kh || !passage_offsets))
    return SKIP_ERR_INVALID_ARG;
  st = check_gate(p, gate);
  if (st != SKIP_OK) return st;
  const size_t need = workspace_size(*p) + gate_scratch_bytes(*p, gate->hidden);
  if (workspace_bytes < need) return SKIP_ERR_WORKSPACE;
  if (p->total_passages == 0) return SKIP_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Workspace w = carve_workspace(*p, workspace);
  GateScratch g = carve_gate_scratch(*p, gate->hidden, static_cast<char*>(workspace) + w.bytes);
  // the passage keys when they are not given, then q_bar, v_bar and the
  // gate inputs, then the gate
  if (!passage_keys) SKIP_TRY(launch_passage_keys(*p, Kh, passage_offsets, w.kbar, s));
  SKIP_TRY(launch_gate_means(*p, Qtok, q_offsets, V_kept, kept_offsets, nullptr, w.kbar,
                             passage_keys, query_passages, g, s));
  SKIP_TRY(launch_gate(*p, *gate, query_passages, g, logits, keep, s));
  return SKIP_OK;
}

// Arguments of the fused route other than the workspace (host-side only).
static skip_status_t check_fused_args(const skip_problem_t* p, const void* V, const void* Qtok,
                                      const int32_t* q_offsets, const void* w_bias,
                                      const int32_t* kept_offsets, const void* Kh,
                                      const void* Vh, const int32_t* passage_offsets,
                                      const int32_t* query_passages,
                                      const float* passage_keys, const int32_t* kept_idx,
                                      const void* O) {
  skip_status_t st = check(p, kPrune | kGraph);
  if (st != SKIP_OK) return st;
  if (!V || !Qtok || !q_offsets || !kept_offsets || !query_passages || !passage_offsets)
    return SKIP_ERR_INVALID_ARG;
  if (p->total_kept > 0 && (!kept_idx || !O)) return SKIP_ERR_INVALID_ARG;
  if (p->total_tokens > 0 && (!Kh || !Vh)) return SKIP_ERR_INVALID_ARG;
  if (!al16(V) || !al16(Qtok) || !al16(w_bias) || !al16(Kh) || !al16(Vh) || !al16(O) ||
      !al16(passage_keys))
    return SKIP_ERR_INVALID_ARG;
  return SKIP_OK;
}

static skip_status_t route_fused_impl(const skip_problem_t* p, const void* V,
                                      const void* Qtok, const int32_t* q_offsets,
                                      const void* w_bias, const int32_t* kept_offsets,
                                      const void* Kh, const void* Vh,
                                      const int32_t* passage_offsets,
                                      const int32_t* query_passages,
                                      const float* passage_keys, int32_t* kept_idx, void* O,
                                      float* lse, void* workspace, size_t workspace_bytes,
                                      void* stream, void* const* ev,
                                      const skip_skv_gate_t* gate = nullptr,
                                      uint8_t* passage_keep = nullptr,
                                      float* gate_logits = nullptr) {
  skip_status_t st = check_fused_args(p, V, Qtok, q_offsets, w_bias, kept_offsets, Kh, Vh,
                                      passage_offsets, query_passages, passage_keys, kept_idx,
                                      O);
  if (st != SKIP_OK) return st;
  if (!workspace) return SKIP_ERR_INVALID_ARG;
  size_t need = workspace_size(*p);
  if (gate) {
    st = check_gate(p, gate);
    if (st != SKIP_OK) return st;
    if (p->total_passages > 0 && !passage_keep) return SKIP_ERR_INVALID_ARG;
    need += gate_scratch_bytes(*p, gate->hidden);
  }
  if (workspace_bytes < need) return SKIP_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Workspace w = carve_workspace(*p, workspace);
  int stage = 0;
  auto mark = [&]() -> hipError_t {
    return ev ? hipEventRecord(static_cast<hipEvent_t>(ev[stage++]), s) : hipSuccess;
  };
  const bool work = p->total_kept > 0;
  QuerySource q{V, kept_idx, p->N};
  SKIP_TRY(mark());
  // question pooling (which also clears the prune launch's counters)
  if (work) SKIP_TRY(launch_pool_question(*p, Qtok, q_offsets, w_bias, w.u, w.counters, s));
  SKIP_TRY(mark());
  // scoring and top-k, with (unless given) the passage-key pooling beside them
  if (work)
    SKIP_TRY(launch_prune(*p, V, w.u, w.z, nullptr, kept_offsets, kept_idx, w.counters, Kh,
                          passage_offsets, passage_keys ? 0 : p->total_passages, w.kbar, s));
  SKIP_TRY(mark());
  if (gate && p->total_passages > 0) {
    // verify step: question and kept-row means with the gate inputs (from
    // the passage keys pooled above), then the gate
    GateScratch g = carve_gate_scratch(*p, gate->hidden, static_cast<char*>(workspace) + w.bytes);
    if (!work && !passage_keys)
      SKIP_TRY(launch_passage_keys(*p, Kh, passage_offsets, w.kbar, s));
    SKIP_TRY(launch_gate_means(*p, Qtok, q_offsets, V, kept_offsets, kept_idx, w.kbar,
                               passage_keys, query_passages, g, s));
    SKIP_TRY(launch_gate(*p, *gate, query_passages, g, gate_logits, passage_keep, s));
  }
  if (work)
    SKIP_TRY(launch_edge_dot(*p, q, kept_offsets, query_passages, w.kbar, passage_keys,
                             EdgePartials{w.part, w.qn2, w.kn2}, s));
  SKIP_TRY(mark());
  // edge selection, with the attention's work list built beside it
  if (work)
    SKIP_TRY(launch_edge_select(*p, EdgePartials{w.part, w.qn2, w.kn2}, kept_offsets,
                                query_passages, w.rowmask, nullptr, nullptr, s,
                                gate ? passage_keep : nullptr, passage_offsets, w.plan));
  SKIP_TRY(mark());
  if (work)
    SKIP_TRY(launch_attention(*p, q, kept_offsets, Kh, Vh, passage_offsets, query_passages,
                              w.rowmask, w.plan, O, lse, s));
  SKIP_TRY(mark());
  return SKIP_OK;
}

skip_status_t skip_route_fused(const skip_problem_t* p, const void* V, const void* Qtok,
                               const int32_t* q_offsets, const void* w_bias,
                               const int32_t* kept_offsets, const void* Kh, const void* Vh,
                               const int32_t* passage_offsets, const int32_t* query_passages,
                               const float* passage_keys, int32_t* kept_idx, void* O,
                               float* lse, void* workspace, size_t workspace_bytes,
                               void* stream) {
  return route_fused_impl(p, V, Qtok, q_offsets, w_bias, kept_offsets, Kh, Vh,
                          passage_offsets, query_passages, passage_keys, kept_idx, O, lse,
                          workspace, workspace_bytes, stream, nullptr);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Route without allocation: the workspace is a file-scope device array.  In
// host code `scratch` names a host-side stand-in, not the device array; its
// device address is looked up once per device (hipGetSymbolAddress, with that
// device current) and only that address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[SKIP_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices];   // device address of `scratch` on each device

// The scratch address on the current device, looked up on first use there.
hipError_t scratch_address(int dev, void** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    g_scratch_dev[dev] = ptr;
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

skip_status_t skip_route_fused_noalloc(const skip_problem_t* p, const void* V, const void* Qtok,
                                       const int32_t* q_offsets, const void* w_bias,
                                       const int32_t* kept_offsets, const void* Kh,
                                       const void* Vh, const int32_t* passage_offsets,
                                       const int32_t* query_passages,
                                       const float* passage_keys, int32_t* kept_idx, void* O,
                                       float* lse, void* stream) {
  // host-side checks first: a problem that does not fit is rejected before
  // any HIP call
  skip_status_t st = check_fused_args(p, V, Qtok, q_offsets, w_bias, kept_offsets, Kh, Vh,
                                      passage_offsets, query_passages, passage_keys, kept_idx,
                                      O);
  if (st != SKIP_OK) return st;
  if (workspace_size(*p) > (size_t)SKIP_NOALLOC_SCRATCH_BYTES) return SKIP_ERR_WORKSPACE;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return SKIP_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return SKIP_ERR_UNSUPPORTED;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (s) {
    int sdev = -1;
    if (hipStreamGetDevice(s, &sdev) != hipSuccess) return SKIP_ERR_INVALID_ARG;
    if (sdev != dev) return SKIP_ERR_INVALID_ARG;
  }
  void* ws = nullptr;
  if (scratch_address(dev, &ws) != hipSuccess) return SKIP_ERR_HIP;
  return route_fused_impl(p, V, Qtok, q_offsets, w_bias, kept_offsets, Kh, Vh,
                          passage_offsets, query_passages, passage_keys, kept_idx, O, lse, ws,
                          (size_t)SKIP_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}

skip_status_t skip_workspace_bytes_regions(const skip_problem_t* p, int32_t r_max,
                                           size_t* bytes) {
  if (!bytes) return SKIP_ERR_INVALID_ARG;
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (r_max < 1 || r_max > 16) return SKIP_ERR_INVALID_ARG;
  *bytes = region_scratch_bytes(*p, r_max);
  return SKIP_OK;
}

skip_status_t skip_region_kmeans(const skip_problem_t* p, const void* rows,
                                 const int32_t* kept_offsets, const int32_t* kept_idx,
                                 int32_t r_max, int32_t n_iter, int32_t* region,
                                 float* centroids, int32_t* sizes, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  skip_status_t st = check_common(p);
  if (st != SKIP_OK) return st;
  if (!kept_offsets || !centroids || !workspace) return SKIP_ERR_INVALID_ARG;
  if (p->total_kept > 0 && (!rows || !region)) return SKIP_ERR_INVALID_ARG;
  if (r_max < 1 || r_max > 16 || n_iter < 1 || n_iter > 1000) return SKIP_ERR_INVALID_ARG;
  if (((uintptr_t)rows & 15) != 0) return SKIP_ERR_INVALID_ARG;
  if (p->k_max > kMaxN) return SKIP_ERR_UNSUPPORTED;
  if (kept_idx) {
    if (p->N < 1 || p->k_max > p->N) return SKIP_ERR_INVALID_ARG;
    if ((int64_t)p->B * p->N > INT32_MAX) return SKIP_ERR_UNSUPPORTED;
  }
  if (workspace_bytes < region_scratch_bytes(*p, r_max)) return SKIP_ERR_WORKSPACE;
  hipStream_t s = static_cast<hipStream_t>(stream);
  SKIP_TRY(launch_regions(*p, rows, kept_offsets, kept_idx, r_max, n_iter, region, centroids,
                          sizes, workspace, s));
  return SKIP_OK;
}

skip_status_t skip_route_fused_gated(const skip_problem_t* p, const skip_skv_gate_t* gate,
                                     const void* V, const void* Qtok,
                                     const int32_t* q_offsets, const void* w_bias,
                                     const int32_t* kept_offsets, const void* Kh,
                                     const void* Vh, const int32_t* passage_offsets,
                                     const int32_t* query_passages,
                                     const float* passage_keys, int32_t* kept_idx,
                                     uint8_t* passage_keep, float* gate_logits, void* O,
                                     float* lse, void* workspace, size_t workspace_bytes,
                                     void* stream) {
  if (!gate) return SKIP_ERR_INVALID_ARG;
  return route_fused_impl(p, V, Qtok, q_offsets, w_bias, kept_offsets, Kh, Vh,
                          passage_offsets, query_passages, passage_keys, kept_idx, O, lse,
                          workspace, workspace_bytes, stream, nullptr, gate, passage_keep,
                          gate_logits);
}

skip_status_t skip_route_fused_profiled(
    const skip_problem_t* p, const void* V, const void* Qtok, const int32_t* q_offsets,
    const void* w_bias, const int32_t* kept_offsets, const void* Kh, const void* Vh,
    const int32_t* passage_offsets, const int32_t* query_passages, const float* passage_keys,
    int32_t* kept_idx, void* O, float* lse, void* workspace, size_t workspace_bytes,
    void* stream, void* const* stage_events, int32_t n_events) {
  if (!stage_events || n_events != SKIP_FUSED_STAGES + 1) return SKIP_ERR_INVALID_ARG;
  for (int i = 0; i < n_events; ++i)
    if (!stage_events[i]) return SKIP_ERR_INVALID_ARG;
  return route_fused_impl(p, V, Qtok, q_offsets, w_bias, kept_offsets, Kh, Vh,
                          passage_offsets, query_passages, passage_keys, kept_idx, O, lse,
                          workspace, workspace_bytes, stream, stage_events);
}

}  // extern "C"

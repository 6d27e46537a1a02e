/*
 * skip.h -- C ABI of the SKIP sparse cross-modal routing core for AMD
 * Instinct MI355X (gfx950).
 *
 * The routing core has two stages (paper: "Salient Knowledge Pathways",
 * Sec. 3.3 and 3.5; App. B.1 and B.3; Alg. 1, scoring/TopK/graph/fuse steps):
 *
 *   1. Question-guided visual pruning (Def. B.1).  For question b with
 *      question tokens Q_b (T_b rows) and visual tokens V_b (N rows):
 *        q_bar_b = mean of the rows of Q_b
 *        z_i     = (q_bar_b / sqrt(d) + w) . v_i        (w: optional content bias)
 *        s_i     = sigmoid(z_i)
 *      and the k_b tokens with the largest z are kept (ties: lowest index
 *      first), reported in ascending index order.
 *
 *   2. Bipartite sparse cross-attention (Def. B.3).  Kept row i of question b
 *      and passage j are joined by an edge when cos(q_i, kbar_j) is among the
 *      E_b = min(ceil(avg_degree * k_b), k_b * P_b) largest cosines of that
 *      question (ties: lower flattened index i * P_b + j first).  q_i is the
 *      row's query vector flattened over heads; kbar_j is the passage key
 *      (the mean of the passage's per-token keys unless passed in).  Two
 *      other cuts and one other compatibility are selectable per call
 *      (skip_edge_rule_t, skip_edge_metric_t).  Then,
 *      per head h, row i attends over every token of its neighbour passages:
 *        e_m = sm_scale * <Qh[i,h], Kh[m,h]>,
 *        O[i,h] = sum_m softmax(e)_m Vh[m,h],  LSE[i,h] = log sum_m exp(e_m).
 *      A row without neighbours gets O = 0 and LSE = -inf.
 *
 * Selection decisions (the kept set and the edge set) are computed from
 * float64 accumulations, so they match a float64 reference on any input whose
 * decisive gap exceeds float64 rounding.  Attention accumulates in float32;
 * in bf16 mode the softmax weights are rounded to bf16 before the PV product.
 *
 * Conventions for every entry point
 *   - The caller owns all memory.  Every array argument is a DEVICE pointer
 *     (global memory of the current HIP device); `p` is a HOST pointer.  The
 *     library allocates no device memory, keeps no state between calls and
 *     may be called concurrently on different streams with different
 *     workspaces.  Calls sharing a workspace must be ordered on one stream.
 *   - Element arrays (V, Qtok, w_bias, Qh, Kh, Vh, O, V_kept) have the element
 *     type given by p->dtype and must be 16-byte aligned; row widths are
 *     multiples of 8 elements.  The float passage_keys table, where given,
 *     must be 16-byte aligned as well (it is read with 16-byte loads).
 *   - Offsets are int32, ascending, starting at 0; offsets arrays are device
 *     arrays whose last entry must equal the matching total in `p`.
 *     Kernels clamp every offset into its declared total, so inconsistent
 *     offsets never cause out-of-bounds access (results are then
 *     unspecified).
 *   - `stream` is a hipStream_t (NULL = the null stream).  Work is enqueued
 *     asynchronously; argument checks happen on the host before anything is
 *     enqueued.  Faults inside kernels surface at the caller's next
 *     synchronisation, as for any HIP call.
 *   - Inputs must be finite.  Same inputs give bitwise-identical outputs on
 *     every call (no floating-point atomics).
 *
 * Errors: SKIP_ERR_INVALID_ARG for a NULL required pointer or inconsistent
 * sizes; SKIP_ERR_UNSUPPORTED for shapes the kernels do not implement (see
 * skip_problem_t); SKIP_ERR_WORKSPACE when workspace_bytes is below
 * skip_workspace_bytes(); SKIP_ERR_HIP when a launch fails.  Nothing is
 * enqueued unless the call returns SKIP_OK.
 */
#ifndef SKIP_H
#define SKIP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SKIP_ABI_VERSION 7

typedef enum skip_status {
  SKIP_OK = 0,
  SKIP_ERR_INVALID_ARG = 1,
  SKIP_ERR_UNSUPPORTED = 2,
  SKIP_ERR_WORKSPACE = 3,
  SKIP_ERR_HIP = 4
} skip_status_t;

typedef enum skip_dtype { SKIP_F32 = 0, SKIP_BF16 = 1 } skip_dtype_t;

/*
 * How the edges of a question's bipartite graph are cut from the k_b x P_b
 * compatibilities c_ij (all rules: ties go to the lower flattened index
 * i * P_b + j, i.e. the lower row, then the lower passage).
 *   SKIP_EDGE_QUESTION_BUDGET  the E_b = min(ceil(avg_degree * k_b), k_b * P_b)
 *                              largest per question: a per-question threshold
 *                              that holds the average degree at avg_degree
 *                              (Def. B.3, threshold set dynamically).
 *   SKIP_EDGE_ROW_TOP          every row keeps its min(ceil(avg_degree), P_b)
 *                              largest (a per-row threshold).
 *   SKIP_EDGE_TOP_FRACTION     the min(ceil(edge_beta * k_b * P_b - 1e-9),
 *                              k_b * P_b) largest per question: top-beta
 *                              sparsity (Sec. 3.5, the quantile form of the
 *                              cut; the 1e-9, in double precision, keeps a
 *                              decimal beta from rounding a whole product up).
 */
typedef enum skip_edge_rule {
  SKIP_EDGE_QUESTION_BUDGET = 0,
  SKIP_EDGE_ROW_TOP = 1,
  SKIP_EDGE_TOP_FRACTION = 2
} skip_edge_rule_t;

/*
 * Compatibility of kept row i and passage j (q_i: the row flattened over
 * heads, width d; kbar_j: the passage key).
 *   SKIP_EDGE_COSINE  cos(q_i, kbar_j), 0 when either norm is 0 (Def. B.3)
 *   SKIP_EDGE_DOT     <q_i, kbar_j> / sqrt(d): the argument of the sigmoid
 *                     of eq. (bsca); the sigmoid is monotone, so cutting on
 *                     the argument keeps the same edges
 * Both are formed from float64 sums.
 */
typedef enum skip_edge_metric { SKIP_EDGE_COSINE = 0, SKIP_EDGE_DOT = 1 } skip_edge_metric_t;

/*
 * Host-side description of one batch of B questions (paper Sec. 3.1 problem
 * statement: visual tokens V, question tokens Q, retrieved passages K).
 *
 * Supported shapes: 1 <= B; 1 <= N <= 16384; d a multiple of 8;
 * H * d_h == d; d_h in {64, 128}; P_max <= 64; k_max * P_max <= 16384
 * (per-question edge candidates); all totals below 2^31 elements.
 */
typedef struct skip_problem {
  int32_t dtype;           /* skip_dtype_t: element type of all element arrays */
  int32_t B;               /* questions in the batch                           */
  int32_t N;               /* visual tokens per question                       */
  int32_t d;               /* embedding width of V, Qtok, Qh rows              */
  int32_t H;               /* attention heads                                  */
  int32_t d_h;             /* head dimension                                   */
  int32_t total_qtok;      /* sum_b T_b = rows of Qtok                         */
  int32_t k_max;           /* max_b k_b                                        */
  int32_t total_kept;      /* sum_b k_b = rows of Qh, O, kept_idx              */
  int32_t P_max;           /* max_b P_b                                        */
  int32_t total_passages;  /* sum_b P_b                                        */
  int32_t total_tokens;    /* sum over passages of their token counts          */
  int32_t L_max;           /* longest passage, in tokens                       */
  int32_t total_edges;     /* length of a caller-given edge_col (else 0)       */
  double avg_degree;       /* target average degree of a kept row (paper: 4)   */
  float sm_scale;          /* logit scale (paper: 1/sqrt(d_h))                 */
  int32_t o_f32;           /* 0: O has the element type of dtype; 1: O is float */
  int32_t edge_rule;       /* skip_edge_rule_t (0: per-question budget)        */
  int32_t edge_metric;     /* skip_edge_metric_t (0: cosine)                   */
  double edge_beta;        /* kept fraction for SKIP_EDGE_TOP_FRACTION, (0, 1] */
} skip_problem_t;

/* ABI version of the loaded library (SKIP_ABI_VERSION). */
int32_t skip_abi_version(void);

/* Static, NUL-terminated description of a status code. */
const char* skip_status_string(skip_status_t s);

/*
 * Workspace size in bytes that every entry point needs for problem `p`
 * (host-only, no device access).  Writes *bytes and returns SKIP_OK, or
 * returns the validation error without writing.
 */
skip_status_t skip_workspace_bytes(const skip_problem_t* p, size_t* bytes);

/*
 * Stage 1: question-guided visual token pruning (Def. B.1; Alg. 1, scoring
 * and TopK steps).
 *   V            [B][N][d]      visual tokens
 *   Qtok         [total_qtok][d] question tokens of all questions
 *   q_offsets    [B+1]          rows of Qtok per question; T_b >= 1 (a
 *                               question with no token is pooled as zero)
 *   w_bias       [d] or NULL    content bias w of Def. B.1
 *   kept_offsets [B+1]          k_b = kept_offsets[b+1] - kept_offsets[b],
 *                               0 <= k_b <= N
 *   kept_idx     out [total_kept] int32 kept token indices in [0, N),
 *                               ascending within each question
 *   scores       out [B][N] float sigmoid scores s_i, or NULL
 *   V_kept       out [total_kept][d] the kept rows of V, or NULL
 */
skip_status_t skip_prune_topk(const skip_problem_t* p, const void* V,
                              const void* Qtok, const int32_t* q_offsets,
                              const void* w_bias, const int32_t* kept_offsets,
                              int32_t* kept_idx, float* scores, void* V_kept,
                              void* workspace, size_t workspace_bytes,
                              void* stream);

/*
 * Main-text salience scorer (Sec. 3.3, eq. qvs): a two-layer perceptron on
 * x_i = [v_i ; q_bar ; v_i (*) q_bar] (width 3d),
 *   a_i = W1 x_i + b1,   s_i = w2 . relu(a_i) + b2,
 * evaluated as the paper's bf16 model would: q_bar enters rounded to bf16
 * (round-to-nearest-even, through float32), the Hadamard term is the bf16
 * rounding of the exact product, products accumulate in float32 (bf16
 * matrix cores) and the second layer sums in float32 then float64.
 *   hidden  h: a multiple of 256, at most 4096
 *   W1      [h][3d] bf16, row j = the weights of hidden unit j: columns
 *           [0, d) weigh v_i, [d, 2d) q_bar, [2d, 3d) v_i (*) q_bar
 *   b1      [h] float, or NULL for zeros
 *   w2      [h] float
 *   b2      output bias
 * The activation is ReLU (the paper does not name one).
 */
typedef struct skip_qvs_mlp {
  int32_t hidden;
  int32_t reserved;        /* must be 0 */
  const void* W1;
  const float* b1;
  const float* w2;
  double b2;
} skip_qvs_mlp_t;

/*
 * Workspace of skip_prune_topk_mlp for problem `p` and hidden width `hidden`
 * (host-only).  Writes *bytes and returns SKIP_OK, or the validation error.
 */
skip_status_t skip_workspace_bytes_mlp(const skip_problem_t* p, int32_t hidden,
                                       size_t* bytes);

/*
 * Stage 1 with the main-text scorer (Sec. 3.3, eq. qvs; Alg. 1, scoring and
 * TopK steps): q_bar pooled as in skip_prune_topk, every visual token scored
 * by the perceptron `mlp` (a HOST pointer to the description; its arrays are
 * device arrays), the k_b tokens of largest s kept (ties: lowest index),
 * reported ascending.  bf16 only (p->dtype == SKIP_BF16, else
 * SKIP_ERR_UNSUPPORTED); d a multiple of 32.
 *   scores   out [B][N] float: the perceptron outputs s_i, or NULL
 * Other arguments as in skip_prune_topk (no content bias: it is a term of the
 * first layer here).  The workspace must hold skip_workspace_bytes_mlp().
 */
skip_status_t skip_prune_topk_mlp(const skip_problem_t* p, const skip_qvs_mlp_t* mlp,
                                  const void* V, const void* Qtok,
                                  const int32_t* q_offsets,
                                  const int32_t* kept_offsets, int32_t* kept_idx,
                                  float* scores, void* V_kept, void* workspace,
                                  size_t workspace_bytes, void* stream);

/*
 * Passage verification gate (App. B.4, Def. B.4; Alg. 1, verify step).  For
 * passage j of question b with embedding e_j (the passage key: the mean of its
 * per-token keys, or passage_keys),
 *   x_j = [q_bar ; v_bar ; e_j ; e_j (*) q_bar ; |e_j - q_bar|]   (width 5d),
 *   logit_j = w2 . relu(W x_j + b1) + b2,   nu_j = sigmoid(logit_j),
 * v_bar the mean of the question's kept visual rows (0 when it has none).
 * Inputs enter as bf16 (q_bar, v_bar, e_j rounded through float32; the
 * product rounded from its exact value; the difference rounded from its
 * float32 value); products accumulate in float32.  The question keeps, among its passages with
 * nu_j >= tau, the ceil(rho * P_b - 1e-9) largest nu (ties: lower index).
 *   hidden  h: a multiple of 64, at most 4096
 *   W       [h][5d] bf16 (blocks in the order of x)
 *   b1      [h] float or NULL;  w2 [h] float;  b2 the output bias
 *   tau     threshold on nu, in (0, 1) (paper: 0.5)
 *   rho     kept fraction of a question's passages, in (0, 1]
 * The activation is ReLU (the paper does not name one).
 */
typedef struct skip_skv_gate {
  int32_t hidden;
  int32_t reserved;        /* must be 0 */
  const void* W;
  const float* b1;
  const float* w2;
  double b2;
  double tau;
  double rho;
} skip_skv_gate_t;

/* Workspace of skip_skv_gate and skip_route_fused_gated for problem `p` and
 * hidden width `hidden`. */
skip_status_t skip_workspace_bytes_gate(const skip_problem_t* p, int32_t hidden,
                                        size_t* bytes);

/*
 * The gate.  V_kept [total_kept][d] are the kept visual rows (as written by
 * skip_prune_topk), Qtok/q_offsets the question tokens, Kh/passage_offsets/
 * query_passages/passage_keys as in skip_bipartite_xattn (passage_keys NULL:
 * pooled from Kh; Kh may then not be NULL).
 *   logits  out [total_passages] float: logit_j, or NULL
 *   keep    out [total_passages] uint8: 1 for a kept passage, else 0; the
 *           cut is taken on the float logits (the values written to logits)
 * bf16 only (SKIP_ERR_UNSUPPORTED otherwise); d a multiple of 32.
 */
skip_status_t skip_skv_gate(const skip_problem_t* p, const skip_skv_gate_t* gate,
                            const void* Qtok, const int32_t* q_offsets,
                            const void* V_kept, const int32_t* kept_offsets,
                            const void* Kh, const int32_t* passage_offsets,
                            const int32_t* query_passages, const float* passage_keys,
                            float* logits, uint8_t* keep, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Learned projection of the kept rows (eq. bsca applies W_v to a kept token
 * and W_k to a chunk before their inner product; Def. B.3 calls them h_v and
 * h_k; the attention query is W_Q v): Y[r] = W x_r for every kept row x_r,
 * gathered as it is read.  bf16 rows and weights, float32 sums on the matrix
 * cores; Y stored as bf16 (round to nearest even) or float.
 *   rows     kept_idx NULL: the kept rows [total_kept][d]; else V [B][N][d],
 *            row r of question b being V[b][kept_idx[r]]
 *   W        [d_out][d] bf16, 16-byte aligned
 *   d_out    a multiple of 256, at most 65536;  d a multiple of 32
 *   Y        out [total_kept][d_out], bf16 (out_f32 = 0) or float (1)
 * bf16 problems only (SKIP_ERR_UNSUPPORTED otherwise).  The workspace holds
 * W repacked for the matrix cores: skip_workspace_bytes_project.
 */
skip_status_t skip_workspace_bytes_project(const skip_problem_t* p, int32_t d_out,
                                           size_t* bytes);
skip_status_t skip_gather_project(const skip_problem_t* p, const void* rows,
                                  const int32_t* kept_offsets, const int32_t* kept_idx,
                                  const void* W, int32_t d_out, void* Y, int32_t out_f32,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * Learned projection of the passage keys (eq. bsca applies W_k to a chunk
 * key; Def. B.3 calls it h_k): keys_out[j] = W k~_j, where k~_j is the
 * bfloat16 rounding (through float) of passage j's key: the caller's
 * passage_keys[j] (float), or, with passage_keys NULL, the mean of the
 * passage's token keys Kh (as pooled for the graph, in double).  bf16
 * weights, float32 sums on the matrix cores, float output; the result is the
 * passage_keys argument of skip_bipartite_xattn_proj when d_out == d.
 *   Kh, passage_offsets  as in skip_bipartite_xattn (unused with passage_keys)
 *   passage_keys  [total_passages][d] float, or NULL; 16-byte aligned
 *   W             [d_out][d] bf16, 16-byte aligned
 *   d_out         a multiple of 256, at most 65536;  d a multiple of 32
 *   keys_out      out [total_passages][d_out] float, 16-byte aligned
 * bf16 problems only (SKIP_ERR_UNSUPPORTED otherwise).  Workspace:
 * skip_workspace_bytes_project_keys (pooled keys, their bf16 rows and W
 * repacked).  Nothing is launched when there are no passages.
 */
skip_status_t skip_workspace_bytes_project_keys(const skip_problem_t* p, int32_t d_out,
                                                size_t* bytes);
skip_status_t skip_project_passage_keys(const skip_problem_t* p, const void* Kh,
                                        const int32_t* passage_offsets,
                                        const float* passage_keys, const void* W,
                                        int32_t d_out, float* keys_out, void* workspace,
                                        size_t workspace_bytes, void* stream);

/*
 * The same projection in two calls, for callers that apply one W to many
 * batches: skip_pack_projection writes W repacked for the matrix cores into a
 * caller buffer of skip_workspace_bytes_project bytes (16-byte aligned), and
 * skip_gather_project_packed multiplies with it, Y bitwise equal to what
 * skip_gather_project gives.  The packed copy is an opaque layout of this
 * ABI version, valid for the d of the problem and the d_out it was packed
 * for; the caller owns it and may reuse it until it changes W.  Errors as for
 * skip_gather_project (a short packed buffer: SKIP_ERR_WORKSPACE).
 */
skip_status_t skip_pack_projection(const skip_problem_t* p, const void* W, int32_t d_out,
                                   void* packed, size_t packed_bytes, void* stream);
skip_status_t skip_gather_project_packed(const skip_problem_t* p, const void* rows,
                                         const int32_t* kept_offsets, const int32_t* kept_idx,
                                         const void* packed, int32_t d_out, void* Y,
                                         int32_t out_f32, void* stream);

/*
 * Regions of the kept tokens (Sec. 3.4: the approximate k-means with which
 * region-conditional retrieval groups the kept tokens before issuing one
 * retrieval query per region centroid; the retrieval is not part of this
 * library).  Question b with k_b kept rows gets R_b = min(floor(k_b / 4),
 * r_max) regions, at least 1 when k_b >= 1 and none when k_b = 0.  Start:
 * centroid r = the kept row at position floor((2r+1) k_b / (2 R_b)) of the
 * question's kept list.  Then n_iter Lloyd iterations in float64: every row to
 * the centroid at the least squared Euclidean distance (ties to the lower
 * region), every centroid to the mean of its rows (a region left without rows
 * keeps its centroid).
 *   rows      kept_idx NULL: the kept rows, [total_kept][d] (as written by
 *             skip_prune_topk); else V [B][N][d], row r of question b being
 *             V[b][kept_idx[r]] (as in the fused route); 16-byte aligned
 *   r_max     1..16 (paper: 8);  n_iter  1..1000;  k_max at most 16384
 *   region    out [total_kept] int32: the region of each kept row after the
 *             last iteration
 *   centroids out [B][r_max][d] float: the centroids after the last
 *             iteration, rounded to float (rows r >= R_b are 0)
 *   sizes     out [B][r_max] int32 rows per region, or NULL
 * Distances are compared as |c_r|^2 - 2 v.c_r (the row's own |v|^2 is common
 * to all regions).  Workspace: skip_workspace_bytes_regions.
 */
skip_status_t skip_workspace_bytes_regions(const skip_problem_t* p, int32_t r_max,
                                           size_t* bytes);
skip_status_t skip_region_kmeans(const skip_problem_t* p, const void* rows,
                                 const int32_t* kept_offsets, const int32_t* kept_idx,
                                 int32_t r_max, int32_t n_iter, int32_t* region,
                                 float* centroids, int32_t* sizes, void* workspace,
                                 size_t workspace_bytes, void* stream);

/*
 * Stage 2: bipartite graph + sparse cross-attention (Def. B.3; Alg. 1,
 * graph and fuse steps) on caller-given kept-row queries.
 *   Qh              [total_kept][H][d_h] queries of the kept rows
 *   kept_offsets    [B+1]
 *   Kh, Vh          [total_tokens][H][d_h] per-token keys and values
 *   passage_offsets [total_passages+1] token offsets; every passage >= 1 token
 *   query_passages  [B+1] passages of question b are
 *                   query_passages[b] .. query_passages[b+1]-1 (P_b may be 0)
 *   passage_keys    [total_passages][d] float passage keys, or NULL to use the
 *                   per-passage mean of Kh
 *   edge_rowptr, edge_col  a caller-given graph (CSR over kept rows, column =
 *                   passage number within the question, p->total_edges
 *                   entries), or both NULL to build the graph by the cosine
 *                   rule; columns outside [0, P_b) are ignored
 *   O               out [total_kept][H][d_h], element type dtype (float if
 *                   p->o_f32)
 *   lse             out [total_kept][H] float natural-log LSE, or NULL
 *   edge_rowptr_out out [total_kept+1] int32, or NULL
 *   edge_col_out    out int32, capacity total_kept * P_max, or NULL; with
 *                   edge_rowptr_out it receives the graph in CSR form
 *                   (columns ascending within a row).  Both or neither.
 */
skip_status_t skip_bipartite_xattn(const skip_problem_t* p, const void* Qh,
                                   const int32_t* kept_offsets, const void* Kh,
                                   const void* Vh,
                                   const int32_t* passage_offsets,
                                   const int32_t* query_passages,
                                   const float* passage_keys,
                                   const int32_t* edge_rowptr,
                                   const int32_t* edge_col, void* O, float* lse,
                                   int32_t* edge_rowptr_out,
                                   int32_t* edge_col_out, void* workspace,
                                   size_t workspace_bytes, void* stream);

/*
 * skip_bipartite_xattn on the verified passages only (Alg. 1: the graph is
 * built over the passages the gate keeps).  passage_keep [total_passages]
 * uint8 (0: dropped) as written by skip_skv_gate: a dropped passage gets no
 * edge, and P_b in every edge budget counts the kept passages of question b.
 * Requires the graph to be built here (edge_rowptr and edge_col NULL).  Other
 * arguments and results as in skip_bipartite_xattn.
 */
skip_status_t skip_bipartite_xattn_masked(const skip_problem_t* p, const void* Qh,
                                          const int32_t* kept_offsets, const void* Kh,
                                          const void* Vh,
                                          const int32_t* passage_offsets,
                                          const int32_t* query_passages,
                                          const float* passage_keys,
                                          const uint8_t* passage_keep, void* O,
                                          float* lse, int32_t* edge_rowptr_out,
                                          int32_t* edge_col_out, void* workspace,
                                          size_t workspace_bytes, void* stream);

/*
 * skip_bipartite_xattn with the graph cut on separate edge rows (eq. bsca:
 * the compatibility of W_v v_i and W_k k_j, while the attention queries are
 * W_Q v_i): the compatibilities are taken between edge_rows and the given
 * passage keys, attention runs on Qh.
 *   edge_rows     [total_kept][d] in the problem's element type (e.g. the
 *                 output of skip_gather_project with W_v)
 *   passage_keys  [total_passages][d] float, required (the keys in the same
 *                 space, e.g. W_k applied to the pooled keys)
 *   passage_keep  NULL or a gate's mask as in skip_bipartite_xattn_masked
 * The graph is built here.  Other arguments and results as in
 * skip_bipartite_xattn.
 */
skip_status_t skip_bipartite_xattn_proj(const skip_problem_t* p, const void* Qh,
                                        const void* edge_rows, const int32_t* kept_offsets,
                                        const void* Kh, const void* Vh,
                                        const int32_t* passage_offsets,
                                        const int32_t* query_passages,
                                        const float* passage_keys,
                                        const uint8_t* passage_keep, void* O, float* lse,
                                        int32_t* edge_rowptr_out, int32_t* edge_col_out,
                                        void* workspace, size_t workspace_bytes,
                                        void* stream);

/*
 * Both stages fused (Alg. 1: scoring, TopK, graph, fuse): the kept visual
 * tokens are the attention queries (Qh = the kept rows of V viewed as
 * [H][d_h], which requires H * d_h == d) and are read straight from V, never
 * written out.  Arguments as in the two calls above.
 */
skip_status_t skip_route_fused(const skip_problem_t* p, const void* V,
                               const void* Qtok, const int32_t* q_offsets,
                               const void* w_bias,
                               const int32_t* kept_offsets, const void* Kh,
                               const void* Vh, const int32_t* passage_offsets,
                               const int32_t* query_passages,
                               const float* passage_keys, int32_t* kept_idx,
                               void* O, float* lse, void* workspace,
                               size_t workspace_bytes, void* stream);

/*
 * Largest scratch (in bytes) that skip_route_fused_noalloc can use: problems
 * whose skip_workspace_bytes() exceeds it are rejected.
 */
#define SKIP_NOALLOC_SCRATCH_BYTES (16u << 20)

/*
 * skip_route_fused for callers that cannot allocate device memory (code under
 * HIP graph capture, serving loops, harnesses that forbid hipMalloc): the
 * same route, results bitwise equal to skip_route_fused, with the workspace
 * taken from a buffer of SKIP_NOALLOC_SCRATCH_BYTES bytes that the library
 * holds in device memory on every GPU it is loaded on, until the process
 * ends.  The call allocates and frees nothing.
 *   - The problem's skip_workspace_bytes() must not exceed
 *     SKIP_NOALLOC_SCRATCH_BYTES, else SKIP_ERR_WORKSPACE (nothing enqueued).
 *   - The buffer is per GPU and shared by every call on that GPU: calls on
 *     one GPU whose executions overlap (different streams, or host threads
 *     with no ordering between them) race on it and give unspecified
 *     results.  Order them, e.g. on one stream.  The buffer keeps what the
 *     last call left; every value the route reads is written by the same
 *     call first, so nothing needs clearing between calls.
 *   - `stream` must belong to the current device (SKIP_ERR_INVALID_ARG
 *     otherwise); the first call on a device looks up the buffer's address
 *     there (SKIP_ERR_HIP if that fails).
 * Other arguments and results as in skip_route_fused.
 */
skip_status_t skip_route_fused_noalloc(const skip_problem_t* p, const void* V,
                                       const void* Qtok, const int32_t* q_offsets,
                                       const void* w_bias, const int32_t* kept_offsets,
                                       const void* Kh, const void* Vh,
                                       const int32_t* passage_offsets,
                                       const int32_t* query_passages,
                                       const float* passage_keys, int32_t* kept_idx,
                                       void* O, float* lse, void* stream);

/* Kernel stages of skip_route_fused, in launch order: question pooling;
 * salience scoring with the top-k (and the passage-key pooling unless the
 * keys are given) in one launch; edge compatibilities (partial dot products
 * over slices of d); edge selection (the candidates' keys from the slice
 * sums, then the selection with the attention's work list built beside it);
 * attention. */
#define SKIP_FUSED_STAGES 5

/*
 * skip_route_fused with per-stage timing, for profiling harnesses.
 * stage_events holds n_events == SKIP_FUSED_STAGES + 1 hipEvent_t handles
 * created by the caller (host array of handles); event s is recorded on
 * `stream` just before stage s is enqueued and the last one after the final
 * stage, so hipEventElapsedTime(events[s], events[s+1]) is the duration of
 * stage s.  The stages, in order, as listed for SKIP_FUSED_STAGES:
 * question pooling; scoring with the top-k and (unless the caller gives
 * passage keys) the passage-key pooling; edge compatibilities (in the gated
 * route preceded by the gate); edge selection; attention.  Other arguments
 * and results as in
 * skip_route_fused; SKIP_ERR_INVALID_ARG if stage_events is NULL or
 * n_events is wrong.
 */
skip_status_t skip_route_fused_profiled(
    const skip_problem_t* p, const void* V, const void* Qtok,
    const int32_t* q_offsets, const void* w_bias, const int32_t* kept_offsets,
    const void* Kh, const void* Vh, const int32_t* passage_offsets,
    const int32_t* query_passages, const float* passage_keys,
    int32_t* kept_idx, void* O, float* lse, void* workspace,
    size_t workspace_bytes, void* stream, void* const* stage_events,
    int32_t n_events);

/*
 * The fused route with the verification step (Alg. 1: scoring, TopK, verify,
 * graph, fuse): skip_route_fused in which the passage gate of skip_skv_gate
 * runs between the top-k and the graph (v_bar the mean of the kept rows of V,
 * read through kept_idx; e_j the passage keys the graph uses) and the graph
 * is built on the verified passages only, as in skip_bipartite_xattn_masked.
 * Workspace: skip_workspace_bytes_gate(p, gate->hidden).
 *   passage_keep out [total_passages] uint8, as written by skip_skv_gate
 *   gate_logits  out [total_passages] float, or NULL
 * bf16 only (SKIP_ERR_UNSUPPORTED otherwise); d a multiple of 32; gate
 * fields as in skip_skv_gate.  Other arguments as in skip_route_fused.
 */
skip_status_t skip_route_fused_gated(const skip_problem_t* p, const skip_skv_gate_t* gate,
                                     const void* V, const void* Qtok,
                                     const int32_t* q_offsets, const void* w_bias,
                                     const int32_t* kept_offsets, const void* Kh,
                                     const void* Vh, const int32_t* passage_offsets,
                                     const int32_t* query_passages,
                                     const float* passage_keys, int32_t* kept_idx,
                                     uint8_t* passage_keep, float* gate_logits, void* O,
                                     float* lse, void* workspace, size_t workspace_bytes,
                                     void* stream);

#ifdef __cplusplus
}
#endif

#endif /* SKIP_H */

"""Plain CPU oracle for the SKIP sparse cross-modal routing core.

TEST INFRASTRUCTURE ONLY.  This module is the checker the GPU path is held
against.  Only the test-suite, the package smoke check and the benchmark's CPU
baseline leg may import or call it; the product path never does, and it
shares no code with the HIP kernels or their host library.

Everything is written for readability, in float64, one question at a time and
one kept row at a time, following the paper's definitions in their own order:

* mean-pooled question embedding (Sec. 3.3; App. B.2, Def. B.2);
* question-guided salience score (App. B.1, Def. B.1; Alg. 1, scoring step)
  with f_q = mean-pool and f_v = identity, plus the optional content bias;
  or the main-text scorer, a two-layer perceptron on [v; q_bar; v * q_bar]
  (Sec. 3.3, eq. qvs) with ReLU and bfloat16 inputs;
* top-k pruning of the visual tokens (Def. B.1; Alg. 1, TopK step);
* the bipartite graph between kept tokens and passages (App. B.3, Def. B.3,
  edge rule; Alg. 1, graph step);
* sparse cross-attention restricted to that graph (Def. B.3, attention rule;
  Alg. 1, fuse step);
* the passage verification gate (App. B.4, Def. B.4; Alg. 1, verify step);
* the regions of the kept tokens, an approximate k-means of them into
  R = min(V'/4, 8) regions (Sec. 3.4, the clustering that feeds per-region
  retrieval; the retrieval itself is not part of this path).

Readings where the paper is silent or inconsistent (each is listed with its
justification in the design notes of the repository):

* selection ranks the pre-sigmoid logit z (sigmoid is monotone, so the kept
  set is the paper's; ranking z avoids spurious saturation ties);
* ties in any top-k go to the lowest index; kept indices are returned in
  ascending order;
* an edge joins a kept visual token and a whole passage; the token attends to
  every token of each neighbour passage;
* the edge threshold is set per question so that exactly
  E = min(ceil(avg_degree * k), k * P) edges survive (the paper sets the edge
  threshold "dynamically" to hold the average degree near 4); ties go to the
  lower flattened index i * P + j.  Two other cuts are available: the top
  beta fraction of a question's pairs (the quantile form of Sec. 3.5) and a
  per-row cut keeping min(ceil(avg_degree), P) passages per row; and one
  other compatibility, the scaled dot product of eq. (bsca) with identity
  projections;
* a passage's key is the mean of its per-token keys over all heads, unless
  the caller supplies passage keys;
* a kept token with no edge gets a zero output and log-sum-exp of -inf;
* all heads share one graph.

Parity pins: every function below is checked in the CPU test-suite against
worked examples, closed forms, brute force on tiny inputs, library routines
for the special cases that reduce to them, and invariants.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np


# --------------------------------------------------------------------------
# Stage 1: question-guided visual salience (Sec. 3.3; App. B.1, Def. B.1)
# --------------------------------------------------------------------------

def mean_pool_question(Q: np.ndarray) -> np.ndarray:
    """q_bar = mean of the T question-token rows (Def. B.2 defines q_bar as
    the mean-pool of Q; Alg. 1 uses it in the difficulty step).  Q: [T, d]."""
    Q = np.asarray(Q, dtype=np.float64)
    if Q.ndim != 2 or Q.shape[0] < 1:
        raise ValueError("need at least one question token")
    return Q.sum(axis=0) / Q.shape[0]


def qvs_logits(V: np.ndarray, q_bar: np.ndarray, w_bias: Optional[np.ndarray] = None) -> np.ndarray:
    """Pre-sigmoid salience z_i = q_bar . v_i / sqrt(d) + w_b . v_i (Def. B.1
    with f_q = mean-pool, f_v = identity).  V: [N, d] -> z: [N]."""
    V = np.asarray(V, dtype=np.float64)
    d = V.shape[1]
    u = np.asarray(q_bar, dtype=np.float64) / math.sqrt(d)
    if w_bias is not None:
        u = u + np.asarray(w_bias, dtype=np.float64)
    return V @ u


def qvs_scores(z: np.ndarray) -> np.ndarray:
    """s_i = sigma(z_i) in [0, 1] (Def. B.1)."""
    z = np.asarray(z, dtype=np.float64)
    return 1.0 / (1.0 + np.exp(-z))


def round_bf16(x) -> np.ndarray:
    """Round to the nearest bfloat16 (ties to even) after a first rounding to
    float32; returned as float64.  bfloat16 keeps the top 16 bits of a float32,
    so rounding adds 0x7fff plus the lowest kept bit and clears the low half
    (inputs are finite)."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    bits = f.view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000
    return bits.astype(np.uint32).view(np.float32).astype(np.float64)


def qvs_mlp_scores(V: np.ndarray, q_bar: np.ndarray, W1: np.ndarray, b1, w2: np.ndarray,
                   b2: float) -> np.ndarray:
    """Main-text salience scorer (Sec. 3.3, eq. qvs): s_i = MLP(v_i || q_bar ||
    v_i * q_bar), a two-layer perceptron with hidden width h:

        a_i = W1 x_i + b1,   s_i = w2 . relu(a_i) + b2,   W1: [h, 3d].

    The model runs in bfloat16 (the paper's mixed precision), so its inputs are
    bfloat16 values: q_bar is rounded once (through float32) and the Hadamard
    term is the bfloat16 rounding of the exact product of two bfloat16 values;
    everything after that is exact here (float64).  V: [N, d] -> s: [N]."""
    V = np.asarray(V, dtype=np.float64)
    N, d = V.shape
    W1 = np.asarray(W1, dtype=np.float64)
    if W1.shape[1] != 3 * d:
        raise ValueError("W1 must be [h, 3d]")
    q = round_bf16(q_bar)                      # [d]
    X3 = round_bf16(V * q[None, :])            # [N, d]
    Wa, Wb, Wc = W1[:, :d], W1[:, d:2 * d], W1[:, 2 * d:]
    A = V @ Wa.T + X3 @ Wc.T + (Wb @ q)[None, :]
    if b1 is not None:
        A = A + np.asarray(b1, dtype=np.float64)[None, :]
    return np.maximum(A, 0.0) @ np.asarray(w2, dtype=np.float64) + float(b2)


def qvs_topk(z: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest logits; among equal logits the lower index
    wins; returned in ascending index order (Def. B.1 keeps ceil(rho L)
    tokens with the highest score; Alg. 1, TopK step)."""
    z = np.asarray(z, dtype=np.float64)
    n = z.shape[0]
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    order = np.lexsort((np.arange(n), -z))     # primary key -z, then index
    return np.sort(order[:k]).astype(np.int64)


def gather_rows(V: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """V_hat = the rows of V at the kept indices (Alg. 1, TopK step)."""
    return np.asarray(V)[np.asarray(idx, dtype=np.int64)]


def project_rows(X: np.ndarray, W: np.ndarray) -> np.ndarray:
    """Learned projection of rows, y_i = W x_i (eq. bsca applies W_v to a
    kept token and W_k to a chunk before their inner product; Def. B.3 names
    them h_v and h_k; the attention query is W_Q v).  X: [n, d], W: [d_out,
    d] -> [n, d_out], float64."""
    X = np.asarray(X, dtype=np.float64)
    W = np.asarray(W, dtype=np.float64)
    if X.shape[1] != W.shape[1]:
        raise ValueError("W must be [d_out, d]")
    return X @ W.T


# --------------------------------------------------------------------------
# Regions of the kept tokens (Sec. 3.4, region-conditional retrieval)
# --------------------------------------------------------------------------

def region_count(k: int, r_max: int = 8) -> int:
    """R = min(V'/4, 8) regions for V' = k kept tokens (Sec. 3.4), V'/4 taken
    down to a whole number, at least one region when any token is kept and
    none when none is; r_max replaces the 8."""
    if k <= 0:
        return 0
    return max(1, min(k // 4, int(r_max)))


def region_kmeans(Vhat: np.ndarray, R: int, n_iter: int):
    """Approximate k-means of the kept rows in embedding space (Sec. 3.4):
    a fixed number of Lloyd iterations from a fixed start.

    * start: centroid r is the kept row at position floor((2r+1) k / (2R)) of
      the kept list, the middle of the r-th of R equal runs of it (the list is
      in ascending token order, so the runs are spread over the image);
    * iteration: every row goes to the centroid at the least squared
      Euclidean distance (ties to the lower region), then every centroid
      becomes the mean of its rows; a region left without rows keeps its
      centroid.

    Vhat: [k, d].  Returns (assignment [k] int, centroids [R, d] float64,
    sizes [R] int) after n_iter iterations."""
    X = np.asarray(Vhat, dtype=np.float64)
    k = X.shape[0]
    if R < 1 or R > k:
        raise ValueError("need 1 <= R <= k")
    if n_iter < 1:
        raise ValueError("need at least one iteration")
    C = np.stack([X[((2 * r + 1) * k) // (2 * R)] for r in range(R)])
    assign = np.zeros(k, dtype=np.int64)
    for _ in range(n_iter):
        for i in range(k):
            dist = ((X[i][None, :] - C) ** 2).sum(axis=1)
            assign[i] = int(np.argmin(dist))        # first minimum: the lower region
        for r in range(R):
            members = X[assign == r]
            if members.shape[0] > 0:
                C[r] = members.sum(axis=0) / members.shape[0]
    sizes = np.array([int((assign == r).sum()) for r in range(R)], dtype=np.int64)
    return assign, C, sizes


# --------------------------------------------------------------------------
# Stage 2: bipartite graph (App. B.3, Def. B.3, edge rule)
# --------------------------------------------------------------------------

def passage_keys(Kh: np.ndarray, passage_ranges: Sequence[tuple]) -> np.ndarray:
    """k_bar_j = mean over the tokens of passage j of that token's keys,
    flattened over heads.  Kh: [M, H, d_h]; passage_ranges: (start, end)
    token ranges.  Returns [P, H * d_h]."""
    Kh = np.asarray(Kh, dtype=np.float64)
    M = Kh.shape[0]
    flat = Kh.reshape(M, -1)
    out = np.zeros((len(passage_ranges), flat.shape[1]))
    for j, (a, b) in enumerate(passage_ranges):
        if b <= a:
            raise ValueError("a passage needs at least one token")
        out[j] = flat[a:b].sum(axis=0) / (b - a)
    return out


def cosine_matrix(Qrows: np.ndarray, Kbar: np.ndarray) -> np.ndarray:
    """c_ij = cos(q_i, k_bar_j) = <q_i, k_bar_j> / (|q_i| |k_bar_j|), and 0
    when either norm is 0 (Def. B.3 edge rule)."""
    Qrows = np.asarray(Qrows, dtype=np.float64)
    Kbar = np.asarray(Kbar, dtype=np.float64)
    c = np.zeros((Qrows.shape[0], Kbar.shape[0]))
    for i in range(Qrows.shape[0]):
        nq = math.sqrt(float(Qrows[i] @ Qrows[i]))
        for j in range(Kbar.shape[0]):
            nk = math.sqrt(float(Kbar[j] @ Kbar[j]))
            if nq > 0.0 and nk > 0.0:
                c[i, j] = float(Qrows[i] @ Kbar[j]) / (nq * nk)
    return c


def dot_matrix(Qrows: np.ndarray, Kbar: np.ndarray) -> np.ndarray:
    """c_ij = <q_i, k_bar_j> / sqrt(D), D the width of q_i: the argument of
    the sigmoid in the main-text compatibility A_ij (Sec. 3.5, eq. bsca, with
    the projections W_v, W_k taken as the identity or applied by the caller).
    The sigmoid is monotone, so any cut on A_ij is the same cut on c_ij."""
    Qrows = np.asarray(Qrows, dtype=np.float64)
    Kbar = np.asarray(Kbar, dtype=np.float64)
    c = np.zeros((Qrows.shape[0], Kbar.shape[0]))
    scale = 1.0 / math.sqrt(Qrows.shape[1])
    for i in range(Qrows.shape[0]):
        for j in range(Kbar.shape[0]):
            c[i, j] = float(Qrows[i] @ Kbar[j]) * scale
    return c


def compatibility(Qrows: np.ndarray, Kbar: np.ndarray, metric: str = "cosine") -> np.ndarray:
    """Edge compatibilities by name: "cosine" (Def. B.3) or "dot" (eq. bsca)."""
    if metric == "cosine":
        return cosine_matrix(Qrows, Kbar)
    if metric == "dot":
        return dot_matrix(Qrows, Kbar)
    raise ValueError(f"unknown edge metric {metric!r}")


def skv_logits(q_bar: np.ndarray, v_bar: np.ndarray, E: np.ndarray, W: np.ndarray, b1,
               w2: np.ndarray, b2: float) -> np.ndarray:
    """Passage verification (App. B.4, Def. B.4): nu_j = sigma(h(x_j)) with
    x_j = [q_bar; v_bar; e_j; e_j * q_bar; |e_j - q_bar|] and h a two-layer
    perceptron, h(x) = w2 . relu(W x + b1) + b2, W: [h, 5d].  Returns the
    logits h(x_j) (nu is monotone in them).  As for the main-text scorer the
    model takes bfloat16 inputs: q_bar, v_bar and e_j are rounded once (through
    float32), e_j * q_bar is the rounding of the exact product of the rounded
    values and |e_j - q_bar| the rounding of their float32 difference.
    E: [P, d] passage embeddings."""
    E = np.asarray(E, dtype=np.float64)
    P, d = E.shape
    W = np.asarray(W, dtype=np.float64)
    if W.shape[1] != 5 * d:
        raise ValueError("W must be [h, 5d]")
    q = round_bf16(q_bar)
    v = round_bf16(v_bar)
    e = round_bf16(E)
    had = round_bf16(e * q[None, :])
    dif = round_bf16(np.abs(e.astype(np.float32) - q.astype(np.float32)[None, :]))
    X = np.concatenate([np.broadcast_to(q, (P, d)), np.broadcast_to(v, (P, d)), e, had, dif],
                       axis=1)
    A = X @ W.T
    if b1 is not None:
        A = A + np.asarray(b1, dtype=np.float64)[None, :]
    return np.maximum(A, 0.0) @ np.asarray(w2, dtype=np.float64) + float(b2)


def skv_keep(logits: np.ndarray, tau: float, rho: float) -> np.ndarray:
    """Verified passages (Alg. 1, verify step): among the passages with
    nu_j = sigma(logit_j) >= tau, the ceil(rho * P) largest nu (ties to the
    lower index).  sigma is monotone, so nu >= tau is logit >= log(tau / (1 -
    tau)).  Returns a boolean mask [P]."""
    z = np.asarray(logits, dtype=np.float64)
    P = z.shape[0]
    t = math.log(tau) - math.log1p(-tau)
    cap = int(math.ceil(float(rho) * P - 1e-9))
    cand = [j for j in range(P) if z[j] >= t]
    cand.sort(key=lambda j: (-z[j], j))
    keep = np.zeros(P, dtype=bool)
    keep[cand[:cap]] = True
    return keep


def edge_budget(k: int, P: int, avg_degree: float) -> int:
    """E = min(ceil(avg_degree * k), k * P): the number of edges that keeps
    the average degree of a kept token at avg_degree (Def. B.3 sets the edge
    threshold so that the average degree stays near 4); avg_degree >= P
    gives the complete bipartite graph."""
    return int(min(math.ceil(float(avg_degree) * k), k * P))


def fraction_budget(k: int, P: int, beta: float) -> int:
    """E = min(ceil(beta * k * P - 1e-9), k * P): top-beta sparsity, the cut
    at the beta-quantile of the k * P compatibilities (Sec. 3.5).  The 1e-9
    keeps a decimal beta from rounding up a whole product (0.1 * 1920 is
    192.00000000000003 in binary floating point)."""
    return int(min(math.ceil(float(beta) * (k * P) - 1e-9), k * P))


def row_budget(P: int, avg_degree: float) -> int:
    """Edges per row under a per-row cut: min(ceil(avg_degree), P)."""
    return int(min(math.ceil(float(avg_degree)), P))


def bsca_edges(c: np.ndarray, avg_degree: float, rule: str = "question",
               beta: float = 0.1, passage_keep: Optional[np.ndarray] = None) -> np.ndarray:
    """Boolean adjacency [k, P] cut from the compatibilities c (ties to the
    lower flattened index i * P + j under every rule):

    * "question": the edge_budget(k, P, avg_degree) largest of the question
      (Def. B.3 edge rule with a per-question threshold that holds the
      average degree at avg_degree);
    * "fraction": the fraction_budget(k, P, beta) largest of the question
      (top-beta sparsity, Sec. 3.5);
    * "row": each row's row_budget(P, avg_degree) largest (a per-row
      threshold).

    With ``passage_keep`` (the verified passages, Alg. 1 verify step) the
    graph is built on the kept passages only: the others get no edge and P
    in every budget counts kept passages."""
    c = np.asarray(c, dtype=np.float64)
    if passage_keep is not None:
        keep = np.asarray(passage_keep, dtype=bool)
        idx = np.nonzero(keep)[0]
        sub = bsca_edges(c[:, idx], avg_degree, rule, beta)
        adj = np.zeros(c.shape, dtype=bool)
        adj[:, idx] = sub
        return adj
    k, P = c.shape
    if rule == "row":
        D = row_budget(P, avg_degree)
        adj = np.zeros((k, P), dtype=bool)
        for i in range(k):
            order = np.lexsort((np.arange(P), -c[i]))
            adj[i, order[:D]] = True
        return adj
    if rule == "question":
        E = edge_budget(k, P, avg_degree)
    elif rule == "fraction":
        E = fraction_budget(k, P, beta)
    else:
        raise ValueError(f"unknown edge rule {rule!r}")
    flat = c.reshape(-1)
    order = np.lexsort((np.arange(flat.size), -flat))
    adj = np.zeros(flat.size, dtype=bool)
    adj[order[:E]] = True
    return adj.reshape(k, P)


def adjacency_to_csr(adj: np.ndarray):
    """CSR (rowptr [k+1], col [E]) with columns ascending within each row."""
    adj = np.asarray(adj, dtype=bool)
    rowptr = np.zeros(adj.shape[0] + 1, dtype=np.int64)
    cols: List[int] = []
    for i in range(adj.shape[0]):
        js = np.nonzero(adj[i])[0]
        cols.extend(int(j) for j in js)
        rowptr[i + 1] = len(cols)
    return rowptr, np.asarray(cols, dtype=np.int64)


# --------------------------------------------------------------------------
# Stage 3: sparse cross-attention over the graph (Def. B.3, attention rule)
# --------------------------------------------------------------------------

def bsca_attention(Qh: np.ndarray, Kh: np.ndarray, Vh: np.ndarray,
                   passage_ranges: Sequence[tuple], adj: np.ndarray,
                   sm_scale: float, rows: Optional[Sequence[int]] = None,
                   return_probs: bool = False):
    """For every kept row i and head h: e_m = sm_scale * <Qh[i,h], Kh[m,h]>
    over the tokens m of the passages adjacent to row i (in ascending passage
    order), O[i,h] = sum_m softmax(e)_m Vh[m,h], LSE[i,h] = log sum_m exp e_m.
    A row with no neighbour gets O = 0 and LSE = -inf.

    Qh: [k, H, d_h]; Kh, Vh: [M, H, d_h] (this question's tokens);
    passage_ranges: (start, end) into Kh/Vh per passage; adj: [k, P] bool.
    ``rows`` restricts the computation to some kept rows (outputs for other
    rows are left as NaN)."""
    Qh = np.asarray(Qh, dtype=np.float64)
    Kh = np.asarray(Kh, dtype=np.float64)
    Vh = np.asarray(Vh, dtype=np.float64)
    k, H, d_h = Qh.shape
    O = np.full((k, H, d_h), np.nan)
    LSE = np.full((k, H), np.nan)
    probs = {}
    for i in (range(k) if rows is None else rows):
        nbrs = np.nonzero(adj[i])[0]
        if nbrs.size == 0:
            O[i] = 0.0
            LSE[i] = -np.inf
            continue
        idx = np.concatenate([np.arange(*passage_ranges[j]) for j in nbrs])
        for h in range(H):
            Kg = Kh[idx, h, :]                      # [m, d_h]
            Vg = Vh[idx, h, :]
            e = sm_scale * (Kg @ Qh[i, h])          # [m]
            mx = e.max()
            w = np.exp(e - mx)
            den = w.sum()
            p = w / den
            O[i, h] = p @ Vg
            LSE[i, h] = mx + math.log(den)
            if return_probs:
                probs[(i, h)] = p
    if return_probs:
        return O, LSE, probs
    return O, LSE


# --------------------------------------------------------------------------
# Whole route for a batch of questions (Alg. 1: scoring, TopK, graph, fuse)
# --------------------------------------------------------------------------

@dataclass
class RouteResult:
    kept_idx: List[np.ndarray]        # per question, ascending
    z: List[np.ndarray]               # per question logits [N]
    scores: List[np.ndarray]          # per question sigmoid scores [N]
    cos: List[np.ndarray]             # per question [k_b, P_b]
    adj: List[np.ndarray]             # per question [k_b, P_b] bool
    O: List[np.ndarray]               # per question [k_b, H, d_h]
    LSE: List[np.ndarray]             # per question [k_b, H]
    gate_logits: List[np.ndarray] = field(default_factory=list)   # per question [P_b]
    keep: List[np.ndarray] = field(default_factory=list)          # per question [P_b] bool


def _f64(x) -> np.ndarray:
    if hasattr(x, "detach"):          # a torch tensor on the CPU
        import torch
        return x.detach().to(torch.float64).numpy()
    return np.asarray(x, dtype=np.float64)


def route(V, Qtok, q_offsets, kept_offsets, Kh, Vh, passage_offsets,
          query_passages, sm_scale: float, avg_degree: float = 4.0,
          w_bias=None, passage_key_table=None, queries: Optional[Sequence[int]] = None,
          attn_rows: Optional[dict] = None, with_attention: bool = True,
          edge_rule: str = "question", edge_metric: str = "cosine",
          edge_beta: float = 0.1, mlp: Optional[dict] = None,
          gate: Optional[dict] = None) -> RouteResult:
    """Prune, build the graph and attend, question by question.

    V: [B, N, d]; Qtok: [sum T, d]; Kh, Vh: [sum M, H, d_h]; offsets as in
    the library interface.  The attention queries of a kept row are that
    row's visual token viewed as [H, d_h] (identity query projection).
    ``queries`` restricts the work to some questions; ``attn_rows`` maps a
    question to the kept rows whose attention output is wanted.  With
    ``mlp`` (keys W1, b1, w2, b2) the tokens are ranked by the main-text
    scorer instead of the linear logit; the ``z`` and ``scores`` of the
    result are then both the scorer's s.  With ``gate`` (keys W, b1, w2,
    b2, tau, rho) the verification step of Alg. 1 runs between the top-k and
    the graph: v_bar is the mean of the kept rows (0 when there are none),
    e_j the passage keys, and the graph is built on the kept passages only."""
    w = None if w_bias is None else _f64(w_bias)
    pk = None if passage_key_table is None else _f64(passage_key_table)
    B, N, d = V.shape
    H, d_h = Kh.shape[1], Kh.shape[2]
    res = RouteResult([], [], [], [], [], [], [])
    for b in (range(B) if queries is None else queries):
        # inputs are widened to float64 one question at a time
        Q = _f64(Qtok[int(q_offsets[b]):int(q_offsets[b + 1])])
        Vb = _f64(V[b])
        q_bar = mean_pool_question(Q)
        if mlp is None:
            z = qvs_logits(Vb, q_bar, w)
        else:
            z = qvs_mlp_scores(Vb, q_bar, mlp["W1"], mlp.get("b1"), mlp["w2"], mlp["b2"])
        k = int(kept_offsets[b + 1] - kept_offsets[b])
        idx = qvs_topk(z, k)
        Vhat = gather_rows(Vb, idx)
        p0, p1 = int(query_passages[b]), int(query_passages[b + 1])
        t0 = int(passage_offsets[p0]) if p1 > p0 else 0
        ranges = [(int(passage_offsets[j]) - t0, int(passage_offsets[j + 1]) - t0)
                  for j in range(p0, p1)]
        t1 = int(passage_offsets[p1]) if p1 > p0 else 0
        Kq, Vq = _f64(Kh[t0:t1]), _f64(Vh[t0:t1])
        keep = None
        if p1 > p0:
            Kbar = pk[p0:p1] if pk is not None else passage_keys(Kq, ranges)
            if gate is not None:
                v_bar = Vhat.sum(axis=0) / k if k > 0 else np.zeros(d)
                gl = skv_logits(q_bar, v_bar, Kbar, gate["W"], gate.get("b1"), gate["w2"],
                                gate["b2"])
                keep = skv_keep(gl, gate["tau"], gate["rho"])
                res.gate_logits.append(gl)
                res.keep.append(keep)
            c = compatibility(Vhat, Kbar, edge_metric)
            adj = bsca_edges(c, avg_degree, edge_rule, edge_beta, keep)
        else:
            c = np.zeros((k, 0))
            adj = np.zeros((k, 0), dtype=bool)
            if gate is not None:
                res.gate_logits.append(np.zeros(0))
                res.keep.append(np.zeros(0, dtype=bool))
        if with_attention:
            rows = None if attn_rows is None else attn_rows.get(b, [])
            O, LSE = bsca_attention(Vhat.reshape(k, H, d_h), Kq, Vq, ranges, adj,
                                    sm_scale, rows=rows)
        else:
            O, LSE = None, None
        res.kept_idx.append(idx)
        res.z.append(z)
        res.scores.append(qvs_scores(z) if mlp is None else z)
        res.cos.append(c)
        res.adj.append(adj)
        res.O.append(O)
        res.LSE.append(LSE)
    return res


def bipartite_xattn(Qh, kept_offsets, Kh, Vh, passage_offsets, query_passages,
                    sm_scale: float, avg_degree: float = 4.0,
                    passage_key_table=None, adjacency: Optional[List[np.ndarray]] = None,
                    attn_rows: Optional[dict] = None, edge_rule: str = "question",
                    edge_metric: str = "cosine", edge_beta: float = 0.1,
                    passage_keep: Optional[np.ndarray] = None,
                    edge_rows=None):
    """Graph + attention on caller-given kept-row queries Qh [sum k, H, d_h].
    ``adjacency`` (per question [k_b, P_b] bool) replaces the cosine rule
    when the caller brings its own graph.  ``edge_rows`` [sum k, D] (for
    instance W_v v_i, eq. bsca) are the rows the edge compatibilities are
    taken on when they differ from the queries (then the passage keys must
    be given in the same space).  Returns (cos, adj, O, LSE) lists."""
    pk = None if passage_key_table is None else _f64(passage_key_table)
    B = len(kept_offsets) - 1
    H, d_h = Qh.shape[1], Qh.shape[2]
    cos_l, adj_l, O_l, L_l = [], [], [], []
    for b in range(B):
        r0, r1 = int(kept_offsets[b]), int(kept_offsets[b + 1])
        k = r1 - r0
        p0, p1 = int(query_passages[b]), int(query_passages[b + 1])
        t0 = int(passage_offsets[p0]) if p1 > p0 else 0
        t1 = int(passage_offsets[p1]) if p1 > p0 else 0
        ranges = [(int(passage_offsets[j]) - t0, int(passage_offsets[j + 1]) - t0)
                  for j in range(p0, p1)]
        Q = _f64(Qh[r0:r1])
        Erows = Q.reshape(k, H * d_h) if edge_rows is None else _f64(edge_rows[r0:r1])
        Kq, Vq = _f64(Kh[t0:t1]), _f64(Vh[t0:t1])
        if adjacency is not None:
            c = None
            adj = np.asarray(adjacency[b], dtype=bool)
        elif p1 > p0:
            Kbar = pk[p0:p1] if pk is not None else passage_keys(Kq, ranges)
            c = compatibility(Erows, Kbar, edge_metric)
            adj = bsca_edges(c, avg_degree, edge_rule, edge_beta,
                             None if passage_keep is None else passage_keep[p0:p1])
        else:
            c = np.zeros((k, 0))
            adj = np.zeros((k, 0), dtype=bool)
        rows = None if attn_rows is None else attn_rows.get(b, [])
        O, LSE = bsca_attention(Q, Kq, Vq, ranges, adj, sm_scale, rows=rows)
        cos_l.append(c)
        adj_l.append(adj)
        O_l.append(O)
        L_l.append(LSE)
    return cos_l, adj_l, O_l, L_l

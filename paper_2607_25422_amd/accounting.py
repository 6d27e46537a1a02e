"""Algorithmic work of the routing core: bytes and FLOPs the method itself
must move or compute (not the dense work it avoids, not work a kernel wastes
on masked tiles or re-reads).

Attention FLOPs follow the paper's cost model for the sparse cross-attention
(the cost grows with the number of edges times the work per edge; complexity
appendix, FLOPs bound, and the degree-sweep table): every edge (kept row i,
passage j) costs QK^T plus PV over all L_j tokens of passage j in every head,
i.e. 4 * L_j * H * d_h FLOPs.
"""
from __future__ import annotations

import numpy as np


def attention_flops(edge_lengths: np.ndarray, H: int, d_h: int) -> float:
    """edge_lengths: the token count L_j of the passage of every edge."""
    return 4.0 * float(np.sum(edge_lengths, dtype=np.float64)) * H * d_h


def edge_lengths_from_csr(rowptr: np.ndarray, col: np.ndarray, kept_offsets: np.ndarray,
                          query_passages: np.ndarray, passage_offsets: np.ndarray) -> np.ndarray:
    """Token count of the passage behind every edge of a CSR graph whose
    columns are passage numbers within each question."""
    L = np.diff(passage_offsets)
    out = np.empty(int(rowptr[-1]), dtype=np.int64)
    for b in range(len(kept_offsets) - 1):
        r0, r1 = int(kept_offsets[b]), int(kept_offsets[b + 1])
        e0, e1 = int(rowptr[r0]), int(rowptr[r1])
        out[e0:e1] = L[int(query_passages[b]) + col[e0:e1]]
    return out


def touched_passages(rowptr: np.ndarray, col: np.ndarray, kept_offsets: np.ndarray,
                     query_passages: np.ndarray) -> np.ndarray:
    """Global ids of the passages with at least one edge."""
    ids = set()
    for b in range(len(kept_offsets) - 1):
        r0, r1 = int(kept_offsets[b]), int(kept_offsets[b + 1])
        e0, e1 = int(rowptr[r0]), int(rowptr[r1])
        ids.update((int(query_passages[b]) + col[e0:e1]).tolist())
    return np.array(sorted(ids), dtype=np.int64)


def attention_bytes(total_kept: int, d: int, H: int, touched_tokens: int, elem: int,
                    out_elem: int) -> float:
    """Read the kept rows' queries, read K and V of every touched passage
    once, write O and the float32 LSE, read one 8-byte neighbour mask per row."""
    return float(total_kept * d * elem + 2 * touched_tokens * d * elem +
                 total_kept * d * out_elem + total_kept * H * 4 + total_kept * 8)


def score_bytes(B: int, N: int, d: int, elem: int) -> float:
    """The salience pass streams V once (the pooled question is tiny)."""
    return float(B * N * d * elem)


def route_bytes(B: int, N: int, d: int, total_qtok: int, total_kept: int, H: int,
                total_tokens: int, touched_tokens: int, elem: int, pooled_keys: bool) -> float:
    """Whole fused route: V and the question tokens once, K once more for the
    passage keys when they are pooled on the device, the kept rows, K/V of the
    touched passages, O, LSE and the kept indices."""
    b = B * N * d * elem + total_qtok * d * elem
    if pooled_keys:
        b += total_tokens * d * elem
    b += attention_bytes(total_kept, d, H, touched_tokens, elem, elem)
    b += total_kept * 4
    return float(b)

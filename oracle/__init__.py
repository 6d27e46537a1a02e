"""CPU oracle for the SKIP routing core (test infrastructure only: imported
by the test-suite, the package smoke check and the benchmark's CPU baseline,
never by the product path)."""
from .skip_oracle import (  # noqa: F401
    RouteResult, adjacency_to_csr, bipartite_xattn, bsca_attention, bsca_edges,
    compatibility, cosine_matrix, dot_matrix, edge_budget, fraction_budget,
    gather_rows, mean_pool_question, passage_keys, project_rows, qvs_logits, qvs_mlp_scores, qvs_scores,
    qvs_topk, region_count, region_kmeans, round_bf16, route, row_budget, skv_keep,
    skv_logits,
)

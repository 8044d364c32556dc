"""CPU oracle for the LouisKV KV-clustering and retrieval path.

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain, float64 statement
of what the path computes, used to check the HIP implementation.  Only the
tests, the package smoke check and the benchmark's CPU-baseline leg may
import it; the product path never calls it and has no fallback to it.  It
shares no code with the HIP path and imports nothing from it.
"""
from .louiskv_oracle import (
    round_to_bf16,
    round_to_f32,
    squared_distances,
    kmeans_assign,
    kmeans_update,
    kmeans,
    kmeans_finish,
    KMeansResult,
    clustering_cost,
    segment_mean,
    page_units,
    query_similarity,
    boundary_fires,
    stride_fires,
    group_scores,
    select_budget,
    gather_units,
    attention,
)
from .decode_driver import PrefillState, GroupDecoder, prefill_state_from_kmeans, prefill_state_from_pages

__all__ = [
    "round_to_bf16", "round_to_f32", "squared_distances", "kmeans_assign",
    "kmeans_update", "kmeans", "kmeans_finish", "KMeansResult", "clustering_cost",
    "segment_mean", "page_units", "query_similarity", "boundary_fires", "stride_fires",
    "group_scores", "select_budget", "gather_units", "attention",
    "PrefillState", "GroupDecoder", "prefill_state_from_kmeans", "prefill_state_from_pages",
]

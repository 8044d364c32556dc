"""Seeded synthetic inputs for the LouisKV clustering-and-retrieval path.

This package only draws random tensors with the shapes and statistical
structure of the paper's workloads (clustered prompt keys with outlier
channels, temporally local decode queries).  It holds none of the method's
arithmetic: no clustering, scoring, selection or attention.  Both the CPU
oracle's tests and the HIP path's tests and benchmark take their inputs from
here, so the two sides always see the same numbers.
"""
from .workloads import WORKLOADS, Workload, get_workload, tiny_workload
from .gen import (
    seed_for,
    slice_keys_values,
    group_queries,
    seq_queries,
    jump_steps,
    init_indices,
    SliceData,
    make_slices,
)

__all__ = [
    "WORKLOADS", "Workload", "get_workload", "tiny_workload",
    "seed_for", "slice_keys_values", "group_queries", "seq_queries", "jump_steps",
    "init_indices", "SliceData", "make_slices",
]

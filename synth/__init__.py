"""Seeded synthetic WARP indexes and queries.

This module only draws inputs: centroids, documents, quantised residual codes,
bucket weights and query token embeddings. It holds none of the search path's
arithmetic (no centroid scoring, no lookup tables, no reductions), so both the
CPU oracle and the HIP engine can consume what it produces without sharing any
of the method's code.
"""
from .gen import (  # noqa: F401
    token_vectors,
    with_overrides,
    DIM,
    Workload,
    WORKLOADS,
    SyntheticIndex,
    make_index,
    make_queries,
    pack_codes,
    random_small_workload,
)

"""Seeded synthetic inputs for the paged graph beam search.

This package only *generates* inputs: Gaussian-mixture vectors, the index
graph (sampled-nearest + random edges) and query sets.  It holds none of the
search's own arithmetic and is the only code shared by the CPU oracle side and
the GPU library side (both receive its arrays as plain inputs).
"""
from .gen import (IndexSpec, QuerySpec, Workload, WORKLOADS, build_edges_lib,
                  index_arrays, index_cached, query_array, workload, cache_dir)

__all__ = ["IndexSpec", "QuerySpec", "Workload", "WORKLOADS", "build_edges_lib",
           "index_arrays", "index_cached", "query_array", "workload", "cache_dir"]

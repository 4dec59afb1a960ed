"""Seeded synthetic inputs for the unified AI-query pipeline.

This package only *draws* inputs: columnar tables, token lists, model
weights and query specifications.  It holds none of the method's arithmetic
(no predicate evaluation, no compaction, no transformer math), so that both
the CPU oracle and the GPU harness can consume identical inputs without
sharing any code that computes a result.
"""
from .configs import WORKLOADS, Workload, ModelSpec, TableSpec, query_for, model_spec
from .gen import make_tables, make_model, bf16_round, make_workload

__all__ = [
    "WORKLOADS", "Workload", "ModelSpec", "TableSpec", "query_for", "model_spec",
    "make_tables", "make_model", "bf16_round", "make_workload",
]

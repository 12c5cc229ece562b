"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws numbers: it holds none of the compression method's
arithmetic and imports neither the oracle nor the product library, so both sides
of every parity check can take their inputs from it.
"""
from .gen import (CONFIGS, Config, chunk_rng, gen_rows, gen_all_rows, gnn_batch_ids,
                  dlrm_batch_ids, dlrm_hot_order, structured_rows, micro_rows)

__all__ = ["CONFIGS", "Config", "chunk_rng", "gen_rows", "gen_all_rows", "gnn_batch_ids",
           "dlrm_batch_ids", "dlrm_hot_order", "structured_rows", "micro_rows"]

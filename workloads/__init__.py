"""Seeded synthetic workloads shared by the tests, the benchmark and the oracle's callers."""
from .synth import (CONFIGS, Config, Workload, make_workload, scaled, table_rows,
                    fill_table, torch_dtype, match_stats, zipf_cdf, zipf_tokens,
                    make_fgrams, make_queries, query_batches)

__all__ = ["CONFIGS", "Config", "Workload", "make_workload", "scaled", "table_rows",
           "fill_table", "torch_dtype", "match_stats", "zipf_cdf", "zipf_tokens",
           "make_fgrams", "make_queries", "query_batches"]

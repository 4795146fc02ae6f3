"""MI355X (gfx950) implementation of SCONE's inference-time f-gram embedding path.

The C ABI (include/scone.h, built as libscone.so) holds the hash-table build,
the longest-suffix lookup, the row gather, f-gram discovery and the
precompute of the f-gram rows as HIP kernels; ``scone`` is its
Python binding.
"""
from . import scone
from .scone import (SconeError, Table, HostRows, build_fgram_table, lookup, lookup_counted,
                    gather, embed,
                    embed_pipelined,
                    decode_step, gather_split, split_workspace_bytes, tag, discover_fgrams,
                    discover_workspace_bytes,
                    FgramModel, precompute_fgram_rows, check, check_ok)

__all__ = ["scone", "SconeError", "Table", "HostRows", "build_fgram_table", "lookup", "gather",
           "embed", "embed_pipelined", "decode_step", "gather_split", "split_workspace_bytes", "tag", "discover_fgrams",
           "discover_workspace_bytes",
           "FgramModel", "precompute_fgram_rows", "check",
           "check_ok"]

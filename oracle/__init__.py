"""fp64 CPU oracle (test infrastructure only; never imported by the product path)."""
from .attention import (attn_fwd, attn_bwd, lse_merge, uniform_fwd, uniform_bwd_k0,
                        row_positions, doc_of, default_scale, visible_pairs_bruteforce)

__all__ = ["attn_fwd", "attn_bwd", "lse_merge", "uniform_fwd", "uniform_bwd_k0",
           "row_positions", "doc_of", "default_scale", "visible_pairs_bruteforce"]

"""Float64 CPU oracle (test infrastructure only; never used by the product path)."""
from .relaxkv_oracle import (  # noqa: F401
    Sets, anchor_count, attention_flops, build_sets, score, select, sparse_attn, update_cache,
)

"""Float64 CPU oracle (test infrastructure only; never used by the product path)."""
from .relaxkv_oracle import (  # noqa: F401
    Sets, anchor_count, attention_flops, build_sets, build_sets_context, build_sets_global,
    global_scores, global_scores_f32, global_target_count, query_attn, score, select, select_global, sparse_attn, update_cache,
)

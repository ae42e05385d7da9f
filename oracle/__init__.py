"""CPU oracle (test infrastructure only; see graphattn_oracle)."""
from .graphattn_oracle import (attend, bf16_bits_to_f64, branch_context, branch_slot_ranks,
                               compared_pairs, cosine, decode, equivalence_classes, extend,
                               graph_suffix, is_ancestor, kv_append, kv_copy, kv_head_of, merge,
                               segment_groups, segment_tokens, similarity_margin, state_depths,
                               to_f64)

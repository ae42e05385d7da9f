"""CPU oracle (test infrastructure only; see graphattn_oracle)."""
from .graphattn_oracle import (attend, bf16_bits_to_f64, branch_context, branch_slot_ranks,
                               class_anchor, compared_pairs, correctness_advantage, cosine,
                               decode, efficiency_advantage, equivalence_classes, extend,
                               graph_advantages, graph_suffix, is_ancestor, kv_append, kv_copy,
                               kv_head_of, merge, node_scores, segment_groups, segment_tokens,
                               similarity_margin, state_depths, step_rewards, subtree_outcomes,
                               to_f64)

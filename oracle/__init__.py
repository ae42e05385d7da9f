"""CPU oracle (test infrastructure only; see graphattn_oracle)."""
from .graphattn_oracle import (attend, bf16_bits_to_f64, branch_context, branch_slot_ranks,
                               decode, extend, kv_append, kv_copy, kv_head_of, merge,
                               segment_groups, segment_tokens, to_f64)

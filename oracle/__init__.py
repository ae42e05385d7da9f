"""CPU oracle (test infrastructure only; see graphattn_oracle)."""
from .graphattn_oracle import (attend, bf16_bits_to_f64, branch_context, decode, kv_head_of,
                               merge, segment_groups, branch_slot_ranks, segment_tokens, to_f64)

"""fp64 CPU oracle for MoA attention (test infrastructure only; never on the product path)."""
from .influence_oracle import (block_average_ref, causal_probabilities, grad_wrt_probabilities,
                               influence_profile_ref, influence_ref, influence_rows_ref)
from .search_oracle import (candidate_rules, dominates, masked_pairs, pareto_front_bruteforce, rule_loss_ref,
                            select_bruteforce)
from .moa_oracle import (CacheModel, attention_ref, attention_rows_ref, cache_contents_ref,
                         cache_ref, decode_ref, masked_softmax_rows, plan_ref,
                         probabilities_ref, visible, visible_mask, visible_set, window_ref)

__all__ = [
    "CacheModel", "attention_ref", "attention_rows_ref", "block_average_ref", "cache_contents_ref",
    "cache_ref", "causal_probabilities", "decode_ref", "grad_wrt_probabilities",
    "influence_profile_ref", "influence_ref", "influence_rows_ref", "masked_softmax_rows", "plan_ref",
    "probabilities_ref", "visible", "visible_mask", "visible_set", "window_ref",
    "candidate_rules", "dominates", "masked_pairs", "pareto_front_bruteforce", "rule_loss_ref",
    "select_bruteforce",
]

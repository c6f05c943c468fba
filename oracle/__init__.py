"""CPU oracle of the Hard-KV compression step -- test infrastructure only.

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may use it.
"""
from .hardkv_oracle import *  # noqa: F401,F403
from .hardkv_oracle import (PAGE, MASS_BITS, P_QUANT, logsumexp, read_head, tier_pages,
                            candidate_mask, score_head, redundancy_head, calibrate_head,
                            mix, order_desc, topk_mass, quantise_p, fixed_weight,
                            ToppResult, topp_head, solve_T_head, PageEntry, CompactResult,
                            compact_head, decode_head, merge_states, append_position,
                            pool_max_head, KEEP, SPARSE, REWRITE, score_rows_head,
                            vote_head, budget_plan_head, budget_select_head,
                            compact_mode_head, topk_mass_and_grad, solve_T_gd_head)

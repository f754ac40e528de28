"""fp64 CPU oracle of the RPD commit step (test infrastructure only; the
product path never imports it)."""
from .rpd_oracle import *  # noqa: F401,F403
from .rpd_oracle import (Params, LLADA, DREAM, strict, to_f64, round_to_bf16, final_norm, distribution_stats,
                         project_layer_stats, persistence, confidence_drop, stability_score,
                         candidate_routes, commit_scan, commit_block, commit_closed_form, select,
                         masked_positions, score_commit, layer_stats_masked, assemble, lazy_layer_stats,
                         score_commit_lazy, apply_commit, decode_loop, FLAG_CANDIDATE, FLAG_HIGH_CONF,
                         FLAG_STABLE, FLAG_COMMITTED, FLAG_FALLBACK)

"""CPU oracle of the PISA hot path (test infrastructure; see pisa_oracle)."""
from .pisa_oracle import (  # noqa: F401
    level_sizes, build_pyramid, pyramid_append, lse, score_mean, score_mean_var, SCORES, forced_leaves, select_row, attention_row,
    flat_bsa_row, candidate_score, selection_admissible, flat_bsa_admissible, pyramid_rows, pyramid, select, sparse_attention, select_flat_bsa,
    block_log_mass, selection_quality_row, selection_quality, attention_row_bwd, sparse_attention_bwd,
)

"""Float64 CPU oracle of the DGE eviction step (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never does, and the two
share no code.
"""
from .dge_oracle import *  # noqa: F401,F403
from .dge_oracle import (ROWS_DRAFT, ROWS_WINDOW, ROWS_WINDOW_DRAFT, attention_output,  # noqa: F401
                         cache_attention, causal_probs, compact, evict_layer, evicted_mass,
                         eviction_diagnostics, h2o_colsum,
                         h2o_row_lse, h2o_select, log_partition, maxpool, project_rope, pyramid_budgets,
                         retained_runs, rope, scoring_row_lse, scoring_rows, select_topb, streaming_select, window_scores)

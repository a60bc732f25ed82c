"""fp64 CPU oracle for the Sol-Attn forward pass.

TEST INFRASTRUCTURE: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code with the
GPU library in ``paper_2607_24027_amd``.
"""
from .sol_attn_oracle import (  # noqa: F401
    BAND, MODES, approx_terms, block_counts, diagonal_sigma, exact_logits, exact_terms, forward,
    pool_means, proxy_scores, route, routing, row_stats,
    row_stats_from_moments, thresholds,
)

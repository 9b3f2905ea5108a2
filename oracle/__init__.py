"""CPU oracle of the HGA hot path (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package. The GPU library never does.
"""
from .hga_oracle import (Config, Routing, attend_bwd, attend_fwd, attend_rows_bwd,  # noqa: F401
                         attend_rows_fwd, block_descriptor, candidate_chunks, group_cache_hits, query_descriptor,
                         route, route_rows, routed_tokens, routed_tokens_row, selection_density,
                         summaries, top_k, widen, windows)

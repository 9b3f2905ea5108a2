"""CPU oracle of the HGA hot path (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package. The GPU library never does.
"""
from .hga_oracle import (Config, Routing, attend_bwd, attend_fwd, block_descriptor,  # noqa: F401
                         candidate_chunks, route, routed_tokens, selection_density,
                         summaries, top_k, widen, windows)

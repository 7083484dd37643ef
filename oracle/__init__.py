"""Float64 CPU oracle for the H2O chunk step.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``, never by the library.
"""
from .h2o_oracle import (POLICIES, accumulate_scores, bottomk, decode, elem_err,
                         evict_insert, eviction_agreement,
                         h2o_step, h2o_step_insert_first, kv_gather, kv_scatter, rel_err,
                         sdpa_cache, sdpa_chunk, sdpa_chunk_backward, selection_keys, visible,
                         visible_by_position)

__all__ = ["POLICIES", "accumulate_scores", "bottomk", "decode", "elem_err",
           "evict_insert", "eviction_agreement",
           "h2o_step", "h2o_step_insert_first", "kv_gather", "kv_scatter", "rel_err",
           "sdpa_cache", "sdpa_chunk", "sdpa_chunk_backward", "selection_keys", "visible",
           "visible_by_position"]

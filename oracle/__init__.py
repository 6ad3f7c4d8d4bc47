"""Plain CPU oracle for the sparse-first decode hot path (test infrastructure).

This package is the reference that the HIP path is checked against.  It is
slow on purpose: NumPy in float64, one unit (layer, request, KV head) at a
time, every step written out in the order the paper states it, with no
blocking, fusion or reordering.  bf16 inputs are converted to float64
exactly, so the oracle's only rounding is float64 rounding.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import it.  The product path (``paper_2609_39068_amd``)
never imports, links or calls anything here, and nothing here imports the
product path.

Modules
-------
attention  selected-set attention (Appendix A.1, eq. background-selected-attention)
           with the GQA head map (Appendix A.1, "MHA, MQA, and GQA").
h2o        append, accumulated-score update, retention and the compacted
           slot layout (Appendix A.3, eqs. background-h2o-score and
           background-h2o-retention; Section 3.1 "Method-Customized CacheManager").
quest      page summaries, the page upper bound, page selection and the
           sparse decode step (Appendix A.3, eqs. background-quest-summary
           and background-quest-score).
snapkv     SnapKV observation-window scores, max pooling and prompt compaction
           (Appendix A.3, eqs. background-snapkv-score and background-snapkv-retention).
omnikv     OmniKV max-over-heads selection and its reuse by sparse layers
           (Appendix A.3, eqs. background-omnikv-selection and background-omnikv-reuse).
prune      interval prefix-cache pruning (Section 3.2, eq. prefix-pruning;
           Appendix C.2).
brute      independent pure-Python references (dense attention with
           ``math`` only, selection by full ``sorted``) that pin the NumPy
           code on tiny inputs.

Parity status
-------------
Pinned (by brute force, closed forms or the paper's invariants; see
``tests/test_oracle_*.py``): selected attention, score accumulation,
H2O retention, H2O chunk-wise prefill eviction, Quest summaries, Quest
bound, Quest selection, SnapKV scores and pooling, OmniKV selection, interval
pruning.

Parity unpinned by the paper (conventions of this repository, held only by
the oracle): the per-KV-head aggregation of H2O scores and of Quest page
scores under GQA (sum over the group for H2O, max over the group for Quest),
the hole-fill order of the compacted slot layout and the order-keeping slot
layout after interval pruning.  The paper fixes the retained *set* but not
the order of slots after compaction.
"""

from . import attention, brute, h2o, omnikv, prune, quest, snapkv  # noqa: F401

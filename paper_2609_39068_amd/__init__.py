"""Sparse-first decode hot path on MI355X (gfx950): H2O eviction and Quest page
selection around paged GQA decode attention, as HIP kernels behind a C-ABI
(include/sparse_engine.h).  This package holds the HIP sources (csrc/), their
build script, the ctypes binding and the decode-step driver."""

from ._binding import (  # noqa: F401
    EXPORTED, KVView, SparseEngineError, se_accumulate_scores, se_decode_attend, se_decode_step_h2o,
    se_decode_step_h2o_noalloc, se_static_scratch_bytes,
    se_decode_step_quest, se_snapkv_compact, se_omnikv_select, se_attend_slots,
    se_h2o_prefill_chunk, se_prune_interval,
    se_evict_compact, se_quest_select, se_quest_summarize, se_read_device_errors,
    se_version, se_workspace_bytes, status_string, se_probe_read_pages,
    SE_ATTEND_ACCUMULATE, SE_QUEST_SCORES_GIVEN, SE_OP_DECODE_ATTEND, SE_OP_QUEST_SELECT,
    SE_OP_QUEST_STEP, SE_OP_SNAPKV, SE_SNAPKV_SCORE_ONLY, SE_OP_OMNIKV_SELECT, SE_OP_H2O_PREFILL,
    SE_DEVERR_BAD_PAGE, SE_DEVERR_CAPACITY, SE_DEVERR_BAD_LENGTH, SE_DEVERR_BAD_SELECTION,
    SE_DEVERR_BAD_POSITIONS, SE_DEVERR_BAD_INTERVAL,
)
from .decode import H2ODecoder, OmniKVDecoder, QuestDecoder  # noqa: F401

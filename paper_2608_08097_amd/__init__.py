"""OasisKV decode-time hot path on MI355X (gfx950): HIP kernels behind a C ABI.

The kernels live in ``csrc/`` and build into ``liboasis.so`` (see
``build_lib.py``); ``_lib`` is the ctypes binding of ``include/oasis.h`` and
``path`` drives one decode step (score, select, stage, attend) on HIP streams.
"""
from ._lib import (  # noqa: F401
    OasisDims, OasisError, dims, lib, oasis_abi_version, oasis_attn_workspace_bytes,
    oasis_build_summaries, oasis_last_error, oasis_score_blocks, oasis_score_select, oasis_select_topk,
    oasis_sparse_decode_attn, oasis_sparse_decode_attn_noalloc, oasis_stage_blocks, OasisLayerBuffers, oasis_pipeline_create,
    oasis_pipeline_set_layer, oasis_pipeline_step, oasis_pipeline_join, oasis_pipeline_check, oasis_pipeline_set_wait_limit,
    oasis_pipeline_set_prediction_order, PREDICT_AUTO, PREDICT_BESIDE_ATTENTION, PREDICT_AFTER_ATTENTION,
    oasis_pipeline_destroy,
    oasis_pipeline_profile_begin, oasis_pipeline_profile_end, oasis_update_summaries, oasis_copy_blocks,
    oasis_union_selection, oasis_pipeline_set_local_source, oasis_pipeline_set_plan_stream, PLAN_ON_TRANSFER,
    PLAN_ON_PREDICTION, oasis_pipeline_set_fused_prediction, FUSED_PREDICTION_AUTO, FUSED_PREDICTION_OFF,
    FUSED_PREDICTION_ON,
)

"""MI355X-native single pipeline stage of the offloading-based interleaved pipeline.

The compute path is libstage.so (HIP kernels for gfx950 behind the C ABI of
include/stage.h); ``stage`` is its ctypes binding with the same entry points.
"""
from .stage import (  # noqa: F401
    StageConfig, StageLayerWeights, StageError, config_for, lib, EXPORTED, LIB_PATH,
    STAGE_OK, STAGE_EINVAL, STAGE_ENOMEM, STAGE_EHIP, STAGE_ESTATE, STAGE_ERANGE, STAGE_ESLOT,
    STAGE_TIME_CALLS, STAGE_TIME_GATEUP, STAGE_TIME_LAYERS, STAGE_MAX_THRESHOLDS, STAGE_MAX_SEQS_PER_CALL,
    STAGE_MAX_CONTEXT, STAGE_MAX_LANES, stage_decode_lane, stage_prefill_lane, stage_decode_noalloc,
    STAGE_NOALLOC_SCRATCH_BYTES,
    STAGE_RES_OFFLOADED, STAGE_RES_RESIDENT, STAGE_RES_MHA_OFFLOADED, STAGE_RES_MLP_OFFLOADED,
    stage_config_default, stage_init, stage_destroy, stage_load_layer, stage_prefill, stage_decode,
    stage_kv_append, stage_kv_export_tail, stage_reset_sequence, stage_sync, stage_get_block_table,
    stage_kv_park, stage_kv_unpark,
    stage_get_length, stage_get_residency, stage_get_slot_log, stage_get_demotion_log,
    stage_get_timeline, stage_set_timing, stage_get_stats, stage_strerror, stage_get_residency_log,
    stage_plan_offload, StagePlanInput, StagePlanStep, stage_allocate, StageAllocDevice, StageAllocInput,
    StageAllocPlan, STAGE_ALLOC_MAX_DEVICES, STAGE_ALLOC_MAX_LAYERS,
)

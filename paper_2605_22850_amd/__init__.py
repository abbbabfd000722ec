"""MI355X-native layerwise prefix-KV consumption (ObjectCache's GPU hot path).

The compute runs in ``libobjectcache.so`` (hand-written HIP for gfx950, C ABI
in ``include/objectcache.h``); this package only marshals arguments.
"""
from ._lib import (  # noqa: F401
    EXPORTS, LIB_PATH, OC_FAULT_ABORT, OC_FAULT_NONE, OC_FAULT_STALL, OC_FAULT_SHORT_WRITE, OC_MODE_DEVICE_STAGED,
    OC_MODE_HBM_RESIDENT, OC_MODE_PRODUCER, Layout, OcError, Request, lib, oc_abi_version, oc_attention_workspace_bytes,
    oc_block_table_check, oc_context_create, oc_context_destroy, oc_kv_layer_gather, oc_kv_layer_ingest,
    oc_pipeline_last_ms, oc_pipeline_run, oc_suffix_prefill_layer, oc_bandwidth_allocate, ALLOC_POLICIES,
    DELIVERIES, oc_kv_chunks_ingest, oc_kv_chunks_gather, oc_kv_suffix_append, LayerWeights, oc_rest_of_layer,
    oc_suffix_prefill_layer_noalloc, OC_NOALLOC_WORKSPACE_BYTES, oc_epoch_schedule,
)

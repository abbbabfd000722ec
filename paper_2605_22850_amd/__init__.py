"""MI355X-native layerwise prefix-KV consumption (ObjectCache's GPU hot path).

The compute runs in ``libobjectcache.so`` (hand-written HIP for gfx950, C ABI
in ``include/objectcache.h``); this package only marshals arguments.
"""
from ._lib import (  # noqa: F401
    EXPORTS, LIB_PATH, Layout, OcError, lib, oc_abi_version, oc_attention_workspace_bytes, oc_block_table_check,
    oc_kv_layer_gather, oc_kv_layer_ingest, oc_suffix_prefill_layer,
)

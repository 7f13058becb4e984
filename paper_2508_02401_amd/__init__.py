"""MI355X-native CompressKV prefill-end KV eviction (arXiv 2508.02401).

The path runs in libckv.so (HIP kernels for gfx950 behind the C ABI declared in
include/ckv.h); this package is its thin Python binding plus seeded synthetic
workloads for tests and benchmarks.
"""
from ._binding import (  # noqa: F401
    CKV_BF16, CKV_F16, CKV_F32, CKV_KEEP_WINDOW, CKV_OK, CKV_SHARE_LAYER, CKV_POOL_AVG, CKV_POOL_MAX,
    CKV_ERR_BUDGET, CKV_ERR_HIP, CKV_ERR_INVALID_ARG, CKV_ERR_MASK, CKV_ERR_UNSUPPORTED,
    CKV_ERR_WORKSPACE, CKV_MAX_SEQS, CKV_NUM_STAGES, EXPORTED, STAGE_NAMES, LIB_PATH, CkvError, Seq, alloc_outputs, alloc_workspace,
    ckv_allocate_budgets, ckv_compress_layer, ckv_compress_stack, ckv_gather, ckv_last_hip_error, ckv_score,
    ckv_select, ckv_set_stack_stage_events, ckv_set_stage_events, ckv_status_string, ckv_workspace_bytes, layer_desc, load,
    attn_desc, kv_cache, ckv_decode_workspace_bytes, ckv_decode_attention, ckv_layer_error_workspace_bytes,
    ckv_layer_error, ckv_normalize_errors, ckv_decode_seq, decode_seq, ckv_decode_batch_workspace_bytes,
    ckv_decode_attention_batch, ckv_streaming_select, snapkv_mask,
    CKV_NOALLOC_MAX_WORKSPACE_BYTES, ckv_compress_layer_noalloc, CKV_STACK_LAYERS_PER_LAUNCH,
    CKV_STACK_CHUNK_TOKENS, stack_layers_per_launch,
)

"""MI355X-native edge-feature join (Connected Content Retriever, §3.1 and §6.3), with the
device sort of the affinity records (Alg. 1 Step 1), the document-id map (§6.3.1, Eq. 6) and
ingestion into the store (§6.2).

The work happens in ``libccjoin.so`` (hand-written HIP kernels for gfx950 behind the C ABI in
``include/cc_join.h``). This package is a thin ctypes binding with the same function names; it
only marshals arguments (device pointers, sizes, the stream) and raises ``CCError`` on a
non-OK status. There is no fallback: if the library is not built, every call raises.
"""
from .binding import (  # noqa: F401
    CCError, PreparedJoin, PreparedJoinBatched, Tuning, cc_join, cc_join_batched, cc_join_batched_padded, cc_last_device_error,
    cc_sort_affinity, cc_sort_affinity_noalloc, cc_sort_workspace_bytes, cc_status_string,
    SORT_AUTO, SORT_MERGE, SORT_RADIX, SORT_RADIX_MIN_RECORDS,
    cc_store_create, cc_store_destroy, cc_store_info, cc_store_invalid_count,
    cc_store_reset_invalid_count, cc_validate_keys, lib, LIB_PATH, EXPORTS,
    cc_store_create_indexed, cc_upsert_workspace_bytes, cc_store_upsert, cc_resolve_ids,
    cc_store_read, cc_store_layout, cc_set_ingestion_wait_limit,
    CC_ERR_STORE_FULL, CC_ERR_TOO_LARGE, CC_ERR_TIMEOUT,
)

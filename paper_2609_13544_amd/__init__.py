"""MI355X-native error signatures and bit-flip injection (PEAT's hot path).

The work is done by hand-written HIP kernels for gfx950 in libpeat.so
(C ABI: include/peat.h); this package is its thin ctypes binding.
"""
from ._binding import (  # noqa: F401
    BF16, F16, F32, F64, K_INJECT, K_INJECT_SUM, K_SIG_CHUNK, K_SIG_FINALIZE, K_STREAM_READ, K_TOPK_A,
    K_TOPK_B, LIB_PATH, MAX_POSITIONS, MODEL_BITFLIP, MODEL_NAN, MODEL_UNIFORM, MODEL_VALUE, MODEL_ZERO, SIG_BYTES,
    SIG_NP_DTYPE, STREAM_SPAN, cast_round, corrupt_positions, inject_model, PeatError, PreparedItems, PreparedPairs, decode_records, dtype_code,
    finalize_stats, inject, inject_batched, inject_batched_async, lib, profile_enable,
    profile_read, set_stream, signature, signature_batched, signature_batched_async, stream_read,
    strerror, topk_mean, topk_mean_batched, topk_mean_from_signature_batched, topk_mean_mixed_from_signature_batched, series_stats, spearman, normalize_scores,
    signature_mixed, signature_mixed_batched, signature_mixed_batched_async, topk_mean_mixed_batched,
    inject_signature_batched_async, K_SIG_INJECT, NOALLOC_SCRATCH_BYTES, signature_batched_noalloc,
    TOPK_BYTES, decode_topk, topk_mean_batched_async, topk_mean_mixed_batched_async,
    topk_mean_from_signature_batched_async, topk_mean_mixed_from_signature_batched_async, topk_set_entry_capacity,
)

"""MI355X-native prefix-shared beam decode attention (FastTTS hot path).

The compute lives in ``libtts.so`` (HIP for gfx950, C ABI in
``include/tts.h``); ``tts`` is its ctypes binding and ``device`` moves
synthetic workloads into device memory with PyTorch (allocation and
streams only).
"""

from .tts import (  # noqa: F401
    EXPORTED,
    TTSError,
    PrefixMeta,
    load,
    make_desc,
    tts_append_kv,
    tts_build_prefix_meta,
    tts_build_verify_meta,
    tts_copy_blocks,
    tts_fork_prefix_meta,
    tts_fork_tables,
    tts_kv_alloc_search,
    tts_kv_alloc_time,
    tts_prefix_schedule,
    tts_truncated_lengths,
    tts_prefix_verify_attn,
    tts_paged_decode_attn,
    tts_paged_decode_workspace_size,
    tts_prefix_decode_attn,
    tts_prefix_decode_attn_noalloc,
    tts_prefix_decode_merge,
    tts_prefix_decode_partials,
    tts_prefix_decode_workspace_size,
    tts_prefix_meta_coverage,
    tts_prefix_meta_destroy,
    tts_prefix_meta_export,
    tts_prefix_meta_stats,
    tts_plan_units_host,
)

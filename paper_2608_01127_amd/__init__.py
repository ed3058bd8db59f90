"""MI355X-native block-causal attention for streaming video world models.

Python face of libmw.so (C ABI in include/mw.h): block-causal multi-head
attention forward/backward (paper Sec. 3.2), the ring-buffered rolling KV
cache and cached attention of queued in-flight chunks, and the host plan of
the pipelined denoiser (paper Sec. 3.5), and an fp8 (e4m3) variant of the
cached attention for inference (the quantization direction of Sec. 6).
The functions carry the C entry points' names; all compute runs in the HIP
kernels of csrc/.
"""
from ._lib import (  # noqa: F401
    KVCache,
    MWError,
    MW_EALIGN,
    MW_EEMPTY,
    MW_EFULL,
    MW_EHIP,
    MW_EINVAL,
    MW_EUNSUPPORTED,
    MW_MAX_QUEUED,
    MW_MAX_SLOTS,
    MW_MAX_WINDOW,
    MW_OK,
    MW_QUEUED_CAUSAL,
    MW_QUEUED_ISOLATED,
    load,
    mw_block_causal_attn_bwd,
    mw_block_causal_attn_bwd_noalloc,
    mw_block_causal_attn_bwd_workspace_size,
    mw_block_causal_attn_fwd,
    mw_chunk_attn_cached,
    mw_chunk_attn_cached_fp8,
    mw_chunk_attn_cached_plan,
    mw_chunk_attn_cached_workspace_size,
    mw_kvcache,
    mw_kvcache_append,
    mw_kvcache_evict,
    mw_kvcache_rope_shift,
    mw_kvcache_set_sink,
    mw_rope,
    mw_kvcache_slot_of,
    mw_quantize_fp8,
    mw_sched_config,
    mw_sched_num_ticks,
    mw_sched_plan,
    mw_sched_tick,
    mw_strides,
    sched_config,
)

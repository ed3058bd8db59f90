"""fp64 CPU oracle for block-causal attention and the rolling KV cache.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or call
this package: it exists so that tests, the smoke check and the benchmark's
CPU-baseline leg can check the HIP kernels against a plain, slow, obviously
correct implementation of what the paper defines.  It shares no code with the
HIP path (it imports numpy only).

Contents
- attention.py: block-causal multi-head attention, forward and analytic
  backward, with an explicit mask over all keys (paper Sec. 3.2); cached chunk
  attention for queued in-flight chunks over a window of committed chunks
  (paper Sec. 3.5).
- ring.py: the integer model of the ring-buffered FIFO KV cache
  (paper Sec. 3.5, "Structured Rolling KV Cache").
- rope_rotate (attention.py): rotary position embedding on a band of head
  dimensions, used for the re-shifting of cached keys (paper Sec. 3.5).
- fp8.py: OCP E4M3 encoding, decoding and per-tensor quantization, the
  number format of the fp8 inference variant (the quantization direction the
  paper names in Sec. 6); the fp8 attention itself is checked against
  cached_chunk_attn on the dequantized values.
- scheduler.py: the pipelined asynchronous denoiser simulated tick by tick
  (paper Sec. 3.5, Eq. 4, Eq. 6, Eq. 7): which chunks are in flight, their
  timesteps and updates, commits, evictions and re-shifts.

Parity status: every function here is pinned by the not-gpu tests in
tests/test_oracle.py, tests/test_fp8_oracle.py and tests/test_scheduler.py (library special cases, closed forms, invariants,
finite differences, brute force); none is "parity unpinned".
"""
from .attention import (  # noqa: F401
    chunk_of,
    block_causal_visible,
    attention_fwd,
    attention_bwd,
    block_causal_attn_fwd,
    block_causal_attn_bwd,
    block_causal_attn_fwd_rows,
    cached_visible,
    cached_chunk_attn,
    rope_rotate,
    QUEUED_CAUSAL,
    QUEUED_ISOLATED,
)
from .ring import RingModel, RingError  # noqa: F401
from .fp8 import E4M3_MAX, e4m3_decode, e4m3_encode, quantize_fp8, dequantize_fp8  # noqa: F401
from .scheduler import simulate as simulate_pipeline, shifted_tau, tau_level  # noqa: F401

"""Every entry point launches on the caller's stream (the `stream` argument of the C-ABI, which the
binding takes from torch's current stream): the whole hot path run on a side stream, whose inputs are
written on that stream behind a millisecond of queued work, gives the default-stream results bit for
bit.  A launch on any other stream would race the writes of its inputs."""
import pytest

import synth
from helpers import bits_equal, to_gpu

pytestmark = pytest.mark.gpu


def _path(mw, t, L):
    """Training forward + backward, a bf16 ring (commit, evict, re-shift) with cached attention, and an
    e4m3 ring with quantize-on-commit and its cached attention.  Returns every output."""
    import torch
    B, H, T, D = t["q"].shape
    o, lse = mw.mw_block_causal_attn_fwd(t["q"], t["k"], t["v"], L)
    dq, dk, dv = mw.mw_block_causal_attn_bwd(t["q"], t["k"], t["v"], o, t["do"], lse, L)
    out = [o, lse, dq, dk, dv]
    nc = T // L - 1  # chunks committed; the last one is queued
    qn, kn, vn = (t[n][:, :, nc * L:] for n in ("q", "k", "v"))
    cache = mw.KVCache(nc + 1, B, H, L, D)
    mw.mw_kvcache_set_sink(cache, t["k"][:, :, :64].contiguous(), t["v"][:, :, :64].contiguous())
    for c in range(nc):
        mw.mw_kvcache_append(cache, t["k"][:, :, c * L:(c + 1) * L], t["v"][:, :, c * L:(c + 1) * L])
    mw.mw_kvcache_evict(cache, 1)
    mw.mw_kvcache_rope_shift(cache, 3, 0, 44)
    oc, lc = mw.mw_chunk_attn_cached(qn, kn, vn, 1, L, cache, want_lse=True)
    out += [cache.k_slots[:nc], cache.v_slots[:nc], oc, lc]  # (slot nc is never written)
    c8 = mw.KVCache(nc + 1, B, H, L, D, fp8=True, k_scale=0.02, v_scale=0.02)
    for c in range(nc):
        mw.mw_kvcache_append(c8, t["k"][:, :, c * L:(c + 1) * L], t["v"][:, :, c * L:(c + 1) * L])
    mw.mw_kvcache_evict(c8, 1)
    mw.mw_kvcache_rope_shift(c8, 3, 0, 44)
    q8, k8, v8 = (mw.mw_quantize_fp8(x, 0.02) for x in (qn, kn, vn))
    o8, l8 = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, 1, L, c8, 0.02, want_lse=True)
    out += [c8.k_slots[:nc], c8.v_slots[:nc], q8, o8, l8]
    return [x.view(torch.int16) if x.dtype == torch.bfloat16 else x for x in out]


def test_hot_path_on_a_side_stream(mw):
    import torch
    B, H, T, D, L = 1, 4, 2048, 128, 512
    src = {n: to_gpu(synth.normal_bf16((B, H, T, D), 7100 + i)) for i, n in enumerate(("q", "k", "v", "do"))}
    ref = _path(mw, src, L)
    torch.cuda.synchronize()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        filler = torch.empty(64 << 20, dtype=torch.float32, device="cuda")
        for _ in range(4):  # about a millisecond of work queued ahead of the input writes
            filler.normal_()
        t = {n: torch.empty_like(x).copy_(x) for n, x in src.items()}
        got = _path(mw, t, L)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    assert len(got) == len(ref)
    for i, (a, b) in enumerate(zip(got, ref)):
        assert a.dtype == b.dtype and a.shape == b.shape, i
        assert torch.equal(a, b), f"output {i} differs on the side stream"

"""The attention entry points and the quantizer record into a HIP graph: they allocate nothing when
given their outputs and workspace, set no memory and launch only on the caller's stream.  A captured
training step (forward and backward) and decode step (bf16 and e4m3 cached calls, the e4m3 window with
a re-shift pending, so rotated on load), replayed three times over new inputs with eager work and
synchronizations in between, match eager calls on the same inputs bit for bit on every replay."""
import pytest

import synth
from helpers import to_gpu

pytestmark = pytest.mark.gpu


def test_graph_replay_matches_eager(mw):
    import torch
    B, H, T, D, L, QL = 1, 4, 2048, 128, 512, 64
    bf = dict(dtype=torch.bfloat16, device="cuda")
    x = {n: torch.empty((B, H, T, D), **bf) for n in ("q", "k", "v", "do")}
    qn, kn, vn = (torch.empty((B, H, QL, D), **bf) for _ in range(3))

    def load(seed):
        for i, n in enumerate(("q", "k", "v", "do")):
            x[n].copy_(to_gpu(synth.normal_bf16((B, H, T, D), seed + i)))
        for i, t in enumerate((qn, kn, vn)):
            t.copy_(to_gpu(synth.normal_bf16((B, H, QL, D), seed + 10 + i)))

    # rings filled before capture: the commits, the eviction and the re-shift change the rings' host
    # descriptors and are not recorded; the calls below only read the rings
    cache = mw.KVCache(4, B, H, L, D)
    c8 = mw.KVCache(4, B, H, L, D, fp8=True, k_scale=0.02, v_scale=0.02)
    for c in range(3):
        kc, vc = (to_gpu(synth.normal_bf16((B, H, L, D), 7300 + 2 * c + j)) for j in range(2))
        mw.mw_kvcache_append(cache, kc, vc)
        mw.mw_kvcache_append(c8, kc, vc)
    mw.mw_kvcache_evict(cache, 1)
    mw.mw_kvcache_evict(c8, 1)
    mw.mw_kvcache_rope_shift(c8, 3, 0, 44)  # pending: rotated as each call loads the window

    o = torch.empty_like(x["q"])
    lse = torch.empty((B, H, T), dtype=torch.float32, device="cuda")
    dq, dk, dv = (torch.empty_like(x["q"]) for _ in range(3))
    ws_b = torch.empty(mw.mw_block_causal_attn_bwd_workspace_size(B, H, T, D), dtype=torch.uint8, device="cuda")
    oc, o8 = torch.empty_like(qn), torch.empty_like(qn)
    lc, l8 = (torch.empty((B, H, QL), dtype=torch.float32, device="cuda") for _ in range(2))
    ws_c = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(cache, 1, QL)), dtype=torch.uint8,
                       device="cuda")
    ws_8 = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(c8, 1, QL)), dtype=torch.uint8,
                       device="cuda")
    q8, k8, v8 = (torch.empty((B, H, QL, D), dtype=torch.uint8, device="cuda") for _ in range(3))

    def step():
        mw.mw_block_causal_attn_fwd(x["q"], x["k"], x["v"], L, out=o, lse=lse)
        mw.mw_block_causal_attn_bwd(x["q"], x["k"], x["v"], o, x["do"], lse, L, workspace=ws_b, dq=dq, dk=dk, dv=dv)
        mw.mw_chunk_attn_cached(qn, kn, vn, 1, QL, cache, out=oc, lse=lc, workspace=ws_c)
        for src, dst in ((qn, q8), (kn, k8), (vn, v8)):
            mw.mw_quantize_fp8(src, 0.02, out=dst)
        mw.mw_chunk_attn_cached_fp8(q8, k8, v8, 1, QL, c8, 0.02, out=o8, lse=l8, workspace=ws_8)

    outs = [o, lse, dq, dk, dv, oc, lc, q8, k8, v8, o8, l8]
    load(7400)
    step()  # eager first: split plans memoised, occupancy queried
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()

    for r in range(3):
        load(7500 + 20 * r)
        step()
        torch.cuda.synchronize()
        ref = [t.clone() for t in outs]
        for t in outs:
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(zip(outs, ref)):
            a_, b_ = (a.view(torch.int16), b.view(torch.int16)) if a.dtype == torch.bfloat16 else (a, b)
            assert torch.equal(a_, b_), f"replay {r}: output {i} differs from the eager call"

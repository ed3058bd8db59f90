"""GPU parity at the paper's own shapes (MiniWorld-1B: 12 heads of width 128, chunks of 2 latent
frames x 300 tokens): training over a 32-chunk window, and streaming with 8 in-flight chunks over
a 24-chunk cache and a one-frame sink, with the classifier-free-guidance batch of 2, given to the
kernels as [B,T,H,D] views (the projections' layout)."""
import numpy as np
import pytest

import oracle
import synth
from helpers import assert_close, f64, to_f64, to_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def train_1b(mw):
    import torch
    s = synth.PAPER_1B_TRAIN
    print(f"[case] {s.name} (GPU fwd+bwd)", flush=True)
    bits = synth.training_inputs(s)
    q, k, v, do = (to_gpu(bits[n]) for n in ("q", "k", "v", "do"))
    o, lse = mw.mw_block_causal_attn_fwd(q, k, v, s.chunk_len)
    dq, dk, dv = mw.mw_block_causal_attn_bwd(q, k, v, o, do, lse, s.chunk_len)
    torch.cuda.synchronize()
    return s, bits, {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


def test_paper_1b_training_head_full(train_1b):
    """Head 11 in full: every row and every gradient."""
    s, bits, g = train_1b
    h = 11
    sel = lambda x: x[:, h:h + 1]
    q, k, v, do = (f64(sel(bits[n])) for n in ("q", "k", "v", "do"))
    o, lse = oracle.block_causal_attn_fwd(q, k, v, s.chunk_len, row_block=600)
    assert_close("o", to_f64(g["o"][:, h:h + 1]), o)
    assert_close("lse", to_f64(g["lse"][:, h:h + 1]), lse, max_abs=2e-3, mean_abs=2e-4)
    dq, dk, dv = oracle.block_causal_attn_bwd(q, k, v, do, s.chunk_len, row_block=600)
    for name, ref in (("dq", dq), ("dk", dk), ("dv", dv)):
        assert_close(name, to_f64(g[name][:, h:h + 1]), ref)


def test_paper_1b_training_sampled_rows(train_1b):
    """Every head, sampled rows at chunk edges and the ends, forward."""
    s, bits, g = train_1b
    rows = np.array([0, 599, 600, 1234, 9599, 9600, 18599, 18600, 19199])
    q, k, v = (f64(bits[n]) for n in ("q", "k", "v"))
    go, gl = to_f64(g["o"]), to_f64(g["lse"])
    for h in range(s.H):
        o, lse = oracle.block_causal_attn_fwd_rows(q, k, v, s.chunk_len, 0, h, rows)
        assert_close(f"o rows h{h}", go[0, h, rows], o)
        assert_close(f"lse rows h{h}", gl[0, h, rows], lse, max_abs=2e-3, mean_abs=2e-4)


@pytest.mark.parametrize("window", [24, 12, 6])
def test_paper_1b_streaming_cfg_batch(mw, window):
    """8 in-flight chunks of 600 tokens over `window` cached chunks and a 300-token sink, batch 2
    (conditional + unconditional), inputs and output as [B,T,H,D] views; both batch entries of
    heads 0 and 11 against the oracle."""
    import torch
    s = synth.PAPER_1B_STREAM
    B, H, D, L, nq = s.B, s.H, s.D, s.chunk_len, s.n_queued
    print(f"[case] {s.name} window={window}", flush=True)
    cache = mw.KVCache(window + 1, B, H, L, D)
    hist = [(synth.normal_bf16((B, H, L, D), s.seed_base + 100 + 2 * i),
             synth.normal_bf16((B, H, L, D), s.seed_base + 101 + 2 * i)) for i in range(window + 1)]
    for kc, vc in hist:
        if cache.live == window + 1:
            mw.mw_kvcache_evict(cache, 1)
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    mw.mw_kvcache_evict(cache, 1)
    sk, sv = (synth.normal_bf16((B, H, s.sink_len, D), s.seed_base + 90 + i) for i in range(2))
    gsk, gsv = to_gpu(sk), to_gpu(sv)
    cache.set_sink(gsk, gsv)
    Tq = nq * s.q_len
    inp = {n: synth.normal_bf16((B, Tq, H, D), s.seed_base + 80 + i) for i, n in enumerate(("q", "k", "v"))}
    g = {n: to_gpu(inp[n]).transpose(1, 2) for n in inp}           # [B,H,Tq,D] views of [B,Tq,H,D]
    o_bthd = torch.empty((B, Tq, H, D), dtype=torch.bfloat16, device="cuda")
    o, _ = mw.mw_chunk_attn_cached(g["q"], g["k"], g["v"], nq, s.q_len, cache, out=o_bthd.transpose(1, 2))
    torch.cuda.synchronize()
    win = hist[-window:]
    heads = [(0, 0), (1, 11)]
    bhtd = lambda x: f64(np.ascontiguousarray(np.swapaxes(x, 1, 2)))
    ro, _ = oracle.cached_chunk_attn(bhtd(inp["q"]), bhtd(inp["k"]), bhtd(inp["v"]), [f64(c[0]) for c in win],
                                     [f64(c[1]) for c in win], nq, s.q_len, heads=heads, sink_k=f64(sk),
                                     sink_v=f64(sv))
    go = to_f64(o.contiguous())
    for b, h in heads:
        assert_close(f"o b{b} h{h}", go[b, h], ro[b, h])


def test_paper_05b_training_d72(mw):
    """MiniWorld-0.5B's heads (16 of width 72 = 1152 / 16) over 600-token chunks: two heads in
    full (every row and gradient) and sampled rows of all heads, forward and backward."""
    import torch
    B, H, T, D, L = 1, 16, 4800, 72, 600
    print(f"[case] paper 0.5B training B{B} H{H} T{T} D{D} L{L}", flush=True)
    bits = {n: synth.normal_bf16((B, H, T, D), 8100 + i) for i, n in enumerate(("q", "k", "v", "do"))}
    q, k, v, do = (to_gpu(bits[n]) for n in ("q", "k", "v", "do"))
    o, lse = mw.mw_block_causal_attn_fwd(q, k, v, L)
    dq, dk, dv = mw.mw_block_causal_attn_bwd(q, k, v, o, do, lse, L)
    torch.cuda.synchronize()
    g = {"o": to_f64(o), "lse": to_f64(lse), "dq": to_f64(dq), "dk": to_f64(dk), "dv": to_f64(dv)}
    for h in (0, 15):
        sel = lambda x: x[:, h:h + 1]
        qf, kf, vf, dof = (f64(sel(bits[n])) for n in ("q", "k", "v", "do"))
        ro, rl = oracle.block_causal_attn_fwd(qf, kf, vf, L)
        assert_close(f"o h{h}", g["o"][:, h:h + 1], ro)
        assert_close(f"lse h{h}", g["lse"][:, h:h + 1], rl, max_abs=2e-3, mean_abs=2e-4)
        rdq, rdk, rdv = oracle.block_causal_attn_bwd(qf, kf, vf, dof, L)
        for name, ref in (("dq", rdq), ("dk", rdk), ("dv", rdv)):
            assert_close(f"{name} h{h}", g[name][:, h:h + 1], ref)
    rows = np.array([0, 599, 600, 2999, 4799])
    qa, ka, va = (f64(bits[n]) for n in ("q", "k", "v"))
    for h in range(H):
        ro, rl = oracle.block_causal_attn_fwd_rows(qa, ka, va, L, 0, h, rows)
        assert_close(f"o rows h{h}", g["o"][0, h, rows], ro)


def test_paper_05b_training_bench_shape(mw):
    """The 0.5B training shape exactly as the benchmark times it (B1 H16 T19200 D72, 32 chunks of
    600 tokens): heads 0 and 15 in full, every row of the output and of every gradient."""
    import torch
    B, H, T, D, L = 1, 16, 19200, 72, 600
    print(f"[case] paper 0.5B training bench shape B{B} H{H} T{T} D{D} L{L}", flush=True)
    bits = {n: synth.normal_bf16((B, H, T, D), 8200 + i) for i, n in enumerate(("q", "k", "v", "do"))}
    q, k, v, do = (to_gpu(bits[n]) for n in ("q", "k", "v", "do"))
    o, lse = mw.mw_block_causal_attn_fwd(q, k, v, L)
    dq, dk, dv = mw.mw_block_causal_attn_bwd(q, k, v, o, do, lse, L)
    torch.cuda.synchronize()
    for h in (0, 15):
        sel = lambda x: x[:, h:h + 1]
        qf, kf, vf, dof = (f64(sel(bits[n])) for n in ("q", "k", "v", "do"))
        ro, rl = oracle.block_causal_attn_fwd(qf, kf, vf, L, row_block=600)
        assert_close(f"o h{h}", to_f64(o[:, h:h + 1]), ro)
        assert_close(f"lse h{h}", to_f64(lse[:, h:h + 1]), rl, max_abs=2e-3, mean_abs=2e-4)
        rdq, rdk, rdv = oracle.block_causal_attn_bwd(qf, kf, vf, dof, L, row_block=600)
        for name, got, ref in (("dq", dq, rdq), ("dk", dk, rdk), ("dv", dv, rdv)):
            assert_close(f"{name} h{h}", to_f64(got[:, h:h + 1]), ref)

"""GPU parity of the fp8 (e4m3) inference variant: the quantizer and the quantize-on-commit of
an e4m3 ring bit-exact against oracle/fp8.py, and the e4m3 cached chunk attention (Sec. 3.5
attention, quantized as Sec. 6 suggests) against the fp64 oracle on the dequantized codes."""
import numpy as np
import pytest

import oracle
import synth
from helpers import (FP8_MAX_ABS, FP8_MEAN_ABS, amax_scale, assert_close, bits_equal, f64, to_f64, to_gpu,
                     to_gpu_u8)

pytestmark = pytest.mark.gpu


def sync():
    import torch
    torch.cuda.synchronize()


def codes(bits, scale):
    return oracle.quantize_fp8(synth.bf16_bits_to_f32(bits), scale)


def u8(t):
    return t.detach().cpu().numpy().astype(np.uint8)


@pytest.mark.parametrize("shape,scale,mag,bthd", [
    ((1, 2, 100, 128), 1.0, 1.0, False),
    ((2, 3, 37, 64), 0.0123, 1.0, False),
    ((1, 2, 50, 72), 2.0 ** -5, 4.0, True),        # a [B,T,H,D] view
    ((1, 1, 64, 128), 0.5, 300.0, False),           # many values saturate at +-448 codes
])
def test_quantize_bit_exact(mw, shape, scale, mag, bthd):
    B, H, T, D = shape
    print(f"[case] quantize {shape} scale={scale} mag={mag} bthd={bthd}", flush=True)
    bits = synth.random_bf16(shape, 9100 + T, scale=mag)
    x = to_gpu(bits)
    if bthd:
        x = to_gpu(np.ascontiguousarray(np.swapaxes(bits, 1, 2))).transpose(1, 2)   # [B,H,T,D] view of [B,T,H,D]
    y = mw.mw_quantize_fp8(x, scale)
    sync()
    ref = codes(bits, scale)
    got = u8(y)
    assert got.shape == ref.shape
    assert np.array_equal(got, ref), f"{int((got != ref).sum())} codes differ"


def test_fp8_append_quantizes_into_the_slot(mw):
    """Quantize-on-commit: slot contents bit-exact with the oracle's codes at the cache's scales,
    for contiguous and [B,T,H,D] chunks; the ring bookkeeping is the bf16 ring's."""
    B, H, L, D, S = 1, 3, 80, 128, 3
    ks, vs = 0.013, 0.021
    cache = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    ring = oracle.RingModel(S)
    for i in range(5):
        kb, vb = (synth.normal_bf16((B, H, L, D), 9200 + 2 * i + j) for j in range(2))
        if ring.live == S:
            ring.evict(1)
            mw.mw_kvcache_evict(cache, 1)
        if i % 2:
            kc = to_gpu(np.ascontiguousarray(np.swapaxes(kb, 1, 2))).transpose(1, 2)
            vc = to_gpu(np.ascontiguousarray(np.swapaxes(vb, 1, 2))).transpose(1, 2)
        else:
            kc, vc = to_gpu(kb), to_gpu(vb)
        slot = mw.mw_kvcache_append(cache, kc, vc)
        assert slot == ring.append()
        sync()
        assert np.array_equal(u8(cache.k_slots[slot]), codes(kb, ks))
        assert np.array_equal(u8(cache.v_slots[slot]), codes(vb, vs))
    mw.mw_kvcache_rope_shift(cache, 2, 0, 44)  # e4m3: recorded for rotation on load, the slots stay as committed
    sync()
    assert cache.desc.rope_total == 2 and cache.desc.rope_set == 1
    assert np.array_equal(u8(cache.k_slots[slot]), codes(kb, ks))


def run_fp8_case(mw, B, H, L, S, n_commit, window, nq, qlen, mode, split, sink_len=0, seed=0):
    """Quantize everything on the GPU, run the e4m3 cached attention, return it with the oracle's
    results on the dequantized codes and on the original bf16 values."""
    D = 128
    hist = [(synth.normal_bf16((B, H, L, D), seed + 2 * i), synth.normal_bf16((B, H, L, D), seed + 2 * i + 1))
            for i in range(n_commit)]
    inp = {n: synth.normal_bf16((B, H, nq * qlen, D), seed + 900 + i) for i, n in enumerate(("q", "k", "v"))}
    sink = [synth.normal_bf16((B, H, sink_len, D), seed + 950 + i) for i in range(2)] if sink_len else None
    allk = [c[0] for c in hist] + [inp["k"]] + ([sink[0]] if sink else [])
    allv = [c[1] for c in hist] + [inp["v"]] + ([sink[1]] if sink else [])
    ks = amax_scale(np.concatenate([a.ravel() for a in allk]))
    vs = amax_scale(np.concatenate([a.ravel() for a in allv]))
    qs = amax_scale(inp["q"])
    cache = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    ring = oracle.RingModel(S)
    for kc, vc in hist:
        if ring.live == S:
            ring.evict(1)
            mw.mw_kvcache_evict(cache, 1)
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
        ring.append()
    if sink:
        gsk, gsv = mw.mw_quantize_fp8(to_gpu(sink[0]), ks), mw.mw_quantize_fp8(to_gpu(sink[1]), vs)
        cache.set_sink(gsk, gsv)
    q8 = mw.mw_quantize_fp8(to_gpu(inp["q"]), qs)
    k8 = mw.mw_quantize_fp8(to_gpu(inp["k"]), ks)
    v8 = mw.mw_quantize_fp8(to_gpu(inp["v"]), vs)
    o, lse = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, nq, qlen, cache, qs, window=window, flags=mode, want_lse=True,
                                         split=split)
    sync()
    assert np.array_equal(u8(q8), codes(inp["q"], qs)) and np.array_equal(u8(k8), codes(inp["k"], ks))
    win = ring.window(None if window == -1 else window)
    dq = lambda b, s: oracle.dequantize_fp8(codes(b, s), s)
    ro, rl = oracle.cached_chunk_attn(dq(inp["q"], qs), dq(inp["k"], ks), dq(inp["v"], vs),
                                      [dq(hist[c][0], ks) for c in win], [dq(hist[c][1], vs) for c in win], nq, qlen,
                                      mode=mode, sink_k=dq(sink[0], ks) if sink else None,
                                      sink_v=dq(sink[1], vs) if sink else None)
    rb, _ = oracle.cached_chunk_attn(f64(inp["q"]), f64(inp["k"]), f64(inp["v"]), [f64(hist[c][0]) for c in win],
                                     [f64(hist[c][1]) for c in win], nq, qlen, mode=mode,
                                     sink_k=f64(sink[0]) if sink else None, sink_v=f64(sink[1]) if sink else None)
    return o, lse, ro, rl, rb


@pytest.mark.parametrize("split", [True, False])
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("B,H,L,S,n_commit,window,nq,qlen,sink_len", [
    (1, 2, 96, 4, 6, 3, 2, 96, 0),       # wrapped ring, chunk edges inside tiles
    (2, 1, 160, 5, 5, -1, 3, 160, 0),    # all live chunks, batch 2
    (1, 2, 100, 3, 2, 0, 2, 70, 0),      # empty window: block-causal attention of the queued chunks
    (1, 1, 64, 8, 9, 7, 4, 33, 0),       # short queued chunks
    (1, 2, 120, 4, 4, 3, 3, 120, 40),    # with a sink
    (1, 2, 128, 6, 6, 5, 1, 64, 0),      # one short queued chunk (64-row configuration: two key groups)
    (1, 1, 64, 8, 9, 7, 2, 30, 17),      # 60 rows in two queued chunks, sink of 17, wrapped ring (64-row)
    (1, 2, 96, 3, 4, 2, 1, 7, 0),        # 7 rows over 199 keys: fewer tiles than the pipeline holds
    (1, 2, 128, 6, 6, 5, 1, 100, 32),    # 128-row configuration, ragged
    (1, 1, 300, 3, 1, 1, 3, 300, 0),     # isolated: one whole query tile, the others over 4 key ranges
])
def test_fp8_cached_attention_vs_oracle(mw, split, mode, B, H, L, S, n_commit, window, nq, qlen, sink_len):
    print(f"[case] fp8 cached split={split} mode={mode} B={B} H={H} L={L} S={S} commits={n_commit} w={window} "
          f"nq={nq} qlen={qlen} sink={sink_len}", flush=True)
    o, lse, ro, rl, rb = run_fp8_case(mw, B, H, L, S, n_commit, window, nq, qlen, mode, split, sink_len,
                                      seed=9300 + L + qlen)
    assert_close("o (vs dequantized)", to_f64(o), ro, FP8_MAX_ABS, FP8_MEAN_ABS)
    assert_close("lse", to_f64(lse), rl, max_abs=2e-3, mean_abs=2e-4)
    # end to end (input quantization included) against the unquantized inputs: a looser sanity bar
    assert_close("o (vs bf16 inputs)", to_f64(o), rb, 0.25, 0.025)


def test_fp8_wraparound_invariance_and_determinism(mw):
    """The same window content at two ring offsets gives bit-identical output; reruns too."""
    import torch
    B, H, L, D, nq = 1, 2, 128, 128, 2
    outs = []
    for S, pre in ((4, 0), (5, 3)):
        cache = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=0.01, v_scale=0.01)
        for i in range(pre):     # filler chunks, evicted again, to move the ring offset
            mw.mw_kvcache_append(cache, to_gpu(synth.normal_bf16((B, H, L, D), 9500 + i)),
                                 to_gpu(synth.normal_bf16((B, H, L, D), 9600 + i)))
        mw.mw_kvcache_evict(cache, pre)
        for i in range(3):
            mw.mw_kvcache_append(cache, to_gpu(synth.normal_bf16((B, H, L, D), 9700 + i)),
                                 to_gpu(synth.normal_bf16((B, H, L, D), 9800 + i)))
        q8, k8, v8 = (mw.mw_quantize_fp8(to_gpu(synth.normal_bf16((B, H, nq * L, D), 9900 + i)), 0.01)
                      for i in range(3))
        for _ in range(2):
            o, _ = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, nq, L, cache, 0.01, window=3, split=False)
            outs.append(o.clone())
    sync()
    assert all(bits_equal(outs[0], x) for x in outs[1:])
    assert torch.isfinite(outs[0].float()).all()


@pytest.mark.parametrize("window", [24, 6])
def test_fp8_paper_1b_streaming(mw, window):
    """MiniWorld-1B streaming shape in e4m3: CFG batch 2, 12 heads of 128, 8 in-flight 600-token
    chunks over `window` cached chunks and a 300-token sink; heads (0,0) and (1,11) vs the oracle."""
    import torch
    B, H, D, L, nq, sink_len = 2, 12, 128, 600, 8, 300
    print(f"[case] fp8 paper 1B streaming window={window}", flush=True)
    ks, vs, qs = 0.011, 0.012, 0.0105
    cache = mw.KVCache(window + 1, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    hist = [(synth.normal_bf16((B, H, L, D), 9400 + 2 * i), synth.normal_bf16((B, H, L, D), 9401 + 2 * i))
            for i in range(window)]
    for kc, vc in hist:
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    sk, sv = (synth.normal_bf16((B, H, sink_len, D), 9390 + i) for i in range(2))
    cache.set_sink(mw.mw_quantize_fp8(to_gpu(sk), ks), mw.mw_quantize_fp8(to_gpu(sv), vs))
    inp = {n: synth.normal_bf16((B, H, nq * L, D), 9380 + i) for i, n in enumerate(("q", "k", "v"))}
    q8 = mw.mw_quantize_fp8(to_gpu(inp["q"]), qs)
    k8 = mw.mw_quantize_fp8(to_gpu(inp["k"]), ks)
    v8 = mw.mw_quantize_fp8(to_gpu(inp["v"]), vs)
    o_bthd = torch.empty((B, nq * L, H, D), dtype=torch.bfloat16, device="cuda")
    o, _ = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, nq, L, cache, qs, out=o_bthd.transpose(1, 2))
    sync()
    dq = lambda b, s: oracle.dequantize_fp8(codes(b, s), s)
    heads = [(0, 0), (1, 11)]
    ro, _ = oracle.cached_chunk_attn(dq(inp["q"], qs), dq(inp["k"], ks), dq(inp["v"], vs),
                                     [dq(c[0], ks) for c in hist], [dq(c[1], vs) for c in hist], nq, L, heads=heads,
                                     sink_k=dq(sk, ks), sink_v=dq(sv, vs))
    go = to_f64(o.contiguous())
    for b, h in heads:
        assert_close(f"o b{b} h{h}", go[b, h], ro[b, h], FP8_MAX_ABS, FP8_MEAN_ABS)


@pytest.mark.parametrize("mode", [0, 1])
def test_fp8_stream_config_sampled_heads(mw, mode):
    """The streaming shape the bench times, in e4m3 (4 in-flight 2640-token chunks over a 6-chunk
    window of an 8-slot ring, B1 H16 D128), with the call's own split plan (queued-causal: 32 whole
    query tiles per head, the first chunk's 10 over 3 key ranges); heads 0 and 15 vs the oracle on
    the dequantized codes."""
    s = synth.STREAM
    print(f"[case] fp8 {s.name} mode={mode}", flush=True)
    ks, vs, qs = 0.011, 0.012, 0.0105
    cache = mw.KVCache(s.slots, s.B, s.H, s.chunk_len, s.D, fp8=True, k_scale=ks, v_scale=vs)
    hist = [(synth.normal_bf16((s.B, s.H, s.chunk_len, s.D), 9600 + 2 * i),
             synth.normal_bf16((s.B, s.H, s.chunk_len, s.D), 9601 + 2 * i)) for i in range(s.slots)]
    for kc, vc in hist:  # 8 commits, then keep the newest 6
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    mw.mw_kvcache_evict(cache, s.slots - s.window)
    ns, nw = mw.mw_chunk_attn_cached_plan(cache, s.n_queued, s.q_len, s.window, mode)
    if mode == 0:
        assert (ns, nw) == (3, 32)
    inp = {n: synth.normal_bf16((s.B, s.H, s.n_queued * s.q_len, s.D), 9590 + i) for i, n in enumerate("qkv")}
    q8 = mw.mw_quantize_fp8(to_gpu(inp["q"]), qs)
    k8 = mw.mw_quantize_fp8(to_gpu(inp["k"]), ks)
    v8 = mw.mw_quantize_fp8(to_gpu(inp["v"]), vs)
    o, lse = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, s.n_queued, s.q_len, cache, qs, window=s.window, flags=mode,
                                         want_lse=True)
    sync()
    dq = lambda b, sc: oracle.dequantize_fp8(codes(b, sc), sc)
    win = hist[-s.window:]
    heads = [(0, 0), (0, s.H - 1)]
    ro, rl = oracle.cached_chunk_attn(dq(inp["q"], qs), dq(inp["k"], ks), dq(inp["v"], vs),
                                      [dq(c[0], ks) for c in win], [dq(c[1], vs) for c in win], s.n_queued, s.q_len,
                                      mode=mode, heads=heads)
    go, gl = to_f64(o), to_f64(lse)
    for b, h in heads:
        assert_close(f"o b{b} h{h} plan {(ns, nw)}", go[b, h], ro[b, h], FP8_MAX_ABS, FP8_MEAN_ABS)
        assert_close(f"lse b{b} h{h}", gl[b, h], rl[b, h], max_abs=2e-3, mean_abs=2e-4)


@pytest.mark.parametrize("q_len,shift", [(64, 0), (256, 0), (64, 3), (256, 3)])
def test_fp8_decode_full_window(mw, q_len, shift):
    """The e4m3 cache-bound decode shapes the benchmark times: one queued chunk of q_len tokens
    over the full window of the streaming shape (6 committed 2640-token chunks of an 8-slot ring,
    B1 H16 D128), with the call's own key-range split, with nothing pending and after one
    re-shift of 3 positions (rotated in staging: one query tile per head); every
    head against the oracle on the dequantized codes (the window keys rotated and rounded once)."""
    s = synth.STREAM
    print(f"[case] fp8 decode q_len={q_len} shift={shift} over {s.window} x {s.chunk_len}", flush=True)
    ks, vs, qs = 0.011, 0.012, 0.0105
    cache = mw.KVCache(s.slots, s.B, s.H, s.chunk_len, s.D, fp8=True, k_scale=ks, v_scale=vs)
    hist = [(synth.normal_bf16((s.B, s.H, s.chunk_len, s.D), 9700 + 2 * i),
             synth.normal_bf16((s.B, s.H, s.chunk_len, s.D), 9701 + 2 * i)) for i in range(s.slots + 1)]
    for kc, vc in hist:  # 9 commits: the ring wraps; keep the newest 6
        if cache.live == s.slots:
            mw.mw_kvcache_evict(cache, 1)
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    mw.mw_kvcache_evict(cache, cache.live - s.window)
    if shift:
        mw.mw_kvcache_rope_shift(cache, shift, 0, 44)
    ns, _ = mw.mw_chunk_attn_cached_plan(cache, 1, q_len, s.window)
    inp = {n: synth.normal_bf16((s.B, s.H, q_len, s.D), 9690 + i) for i, n in enumerate("qkv")}
    q8 = mw.mw_quantize_fp8(to_gpu(inp["q"]), qs)
    k8 = mw.mw_quantize_fp8(to_gpu(inp["k"]), ks)
    v8 = mw.mw_quantize_fp8(to_gpu(inp["v"]), vs)
    o, lse = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, 1, q_len, cache, qs, window=s.window, want_lse=True)
    sync()
    dq = lambda b, sc: oracle.dequantize_fp8(codes(b, sc), sc)
    win = hist[-s.window:]
    if shift:  # rotate the committed code values by -shift, round to e4m3 once, scale
        win_k = [oracle.dequantize_fp8(oracle.quantize_fp8(
            oracle.rope_rotate(oracle.dequantize_fp8(codes(c[0], ks), 1.0), -float(shift), 0, 44).astype(np.float32),
            1.0), ks) for c in win]
    else:
        win_k = [dq(c[0], ks) for c in win]
    ro, rl = oracle.cached_chunk_attn(dq(inp["q"], qs), dq(inp["k"], ks), dq(inp["v"], vs),
                                      win_k, [dq(c[1], vs) for c in win], 1, q_len)
    assert_close(f"o q_len={q_len} shift={shift} ({ns} key ranges)", to_f64(o), ro, FP8_MAX_ABS, FP8_MEAN_ABS)
    assert_close("lse", to_f64(lse), rl, max_abs=2e-3, mean_abs=2e-4)


def _reshift_rollout(mw, shifts_per_eviction, steps=6, seed=9800):
    """e4m3 rollout (B1 H2 L96 D128, 4-slot ring, 3-chunk window): commit, evict down to the
    window, then re-shift by the given list of shifts per eviction.  Returns the cache, the
    committed chunks' bits and, per chunk, the shift total pending on it."""
    B, H, L, D, S, W = 1, 2, 96, 128, 4, 3
    ks, vs = 0.011, 0.012
    cache = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    hist, at_commit, total = [], [], 0
    for t in range(steps):
        kb, vb = (synth.normal_bf16((B, H, L, D), seed + 2 * t + j) for j in range(2))
        mw.mw_kvcache_append(cache, to_gpu(kb), to_gpu(vb))
        hist.append((kb, vb))
        at_commit.append(total)
        if cache.live > W:
            mw.mw_kvcache_evict(cache, cache.live - W)
            for sh in shifts_per_eviction:
                mw.mw_kvcache_rope_shift(cache, sh, 0, 44)
                total += sh
    return cache, hist, [total - a for a in at_commit], (B, H, L, D, W, ks, vs)


@pytest.mark.parametrize("mode", [0, 1])
def test_fp8_rope_reshift_on_load_vs_oracle(mw, mode):
    """Re-shift of an e4m3 cache by rotation on load (paper Sec. 3.5, its second option): after a
    rollout with a re-shift of 2 positions per eviction, the attention of two queued chunks equals
    the oracle's over the window keys rotated by each chunk's pending shift and rounded to e4m3
    once (within the fp8 bar), while the slots keep the committed codes bit for bit."""
    cache, hist, pend, (B, H, L, D, W, ks, vs) = _reshift_rollout(mw, [2])
    print(f"[case] fp8 re-shift on load mode={mode} pending={pend[-W:]}", flush=True)
    nq = 2
    inp = {n: synth.normal_bf16((B, H, nq * L, D), 9890 + i) for i, n in enumerate("qkv")}
    qs = 0.0105
    q8, k8, v8 = (mw.mw_quantize_fp8(to_gpu(inp[n]), sc) for n, sc in (("q", qs), ("k", ks), ("v", vs)))
    o, lse = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, nq, L, cache, qs, window=W, flags=mode, want_lse=True)
    sync()
    live = range(len(hist) - W, len(hist))
    for c in live:  # the slots are never rewritten
        assert np.array_equal(u8(cache.k_slots[cache.slot_of(c)]), codes(hist[c][0], ks))
    dq = lambda b, sc: oracle.dequantize_fp8(codes(b, sc), sc)
    win_k = []
    for c in live:  # rotate the committed code values, round to e4m3 once, scale
        vals = oracle.dequantize_fp8(codes(hist[c][0], ks), 1.0)
        rot = oracle.rope_rotate(vals, -float(pend[c]), 0, 44).astype(np.float32)
        win_k.append(oracle.dequantize_fp8(oracle.quantize_fp8(rot, 1.0), ks))
    ro, rl = oracle.cached_chunk_attn(dq(inp["q"], qs), dq(inp["k"], ks), dq(inp["v"], vs), win_k,
                                      [dq(hist[c][1], vs) for c in live], nq, L, mode=mode)
    assert_close("o (rotated on load)", to_f64(o), ro, FP8_MAX_ABS, FP8_MEAN_ABS)
    assert_close("lse", to_f64(lse), rl, max_abs=2e-3, mean_abs=2e-4)


def test_fp8_rope_reshift_pending_total_only(mw):
    """Rotation on load applies each chunk's pending total at once: shifting by 1 three times per
    eviction gives the same output bit for bit as shifting by 3 once, and a shift of +5 then -5
    gives the output of no shift at all (nothing pending, nothing rounded)."""
    outs = []
    for shifts in ([1, 1, 1], [3], [5, -5], []):
        cache, hist, pend, (B, H, L, D, W, ks, vs) = _reshift_rollout(mw, shifts, seed=9900)
        q8, k8, v8 = (mw.mw_quantize_fp8(to_gpu(synth.normal_bf16((B, H, 2 * L, D), 9950 + i)), 0.01)
                      for i in range(3))
        o, _ = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, 2, L, cache, 0.01, window=W)
        outs.append(o.clone())
    sync()
    assert bits_equal(outs[0], outs[1])
    assert bits_equal(outs[2], outs[3])
    assert not bits_equal(outs[1], outs[3])


@pytest.mark.parametrize("q_len,window", [(64, 2), (96, 3)])
def test_fp8_rope_reshift_on_load_sink_partial_window(mw, q_len, window):
    """Rotation on load with a sink (never shifted: it keeps its position), a window smaller than
    the live chunks of a wrapped ring, and a short queued chunk whose call splits the keys (2 and
    3 key ranges at these shapes), so the split partials sit in the workspace after the rotated
    window keys; against the oracle over the window keys rotated by their pending shifts and
    rounded once, fp8 bar."""
    B, H, L, D, S = 1, 2, 256, 128, 4
    ks, vs, qs = 0.011, 0.012, 0.0105
    cache = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    sink_len = 40
    sk, sv = (synth.normal_bf16((B, H, sink_len, D), 9960 + i) for i in range(2))
    cache.set_sink(mw.mw_quantize_fp8(to_gpu(sk), ks), mw.mw_quantize_fp8(to_gpu(sv), vs))
    hist, at_commit, total = [], [], 0
    for t in range(7):  # the ring wraps; each eviction re-shifts by 3
        kb, vb = (synth.normal_bf16((B, H, L, D), 9970 + 2 * t + j) for j in range(2))
        if cache.live == S:
            mw.mw_kvcache_evict(cache, 1)
            mw.mw_kvcache_rope_shift(cache, 3, 0, 44)
            total += 3
        mw.mw_kvcache_append(cache, to_gpu(kb), to_gpu(vb))
        hist.append((kb, vb))
        at_commit.append(total)
    ns, _ = mw.mw_chunk_attn_cached_plan(cache, 1, q_len, window)
    print(f"[case] fp8 re-shift on load q_len={q_len} window={window} splits={ns}", flush=True)
    inp = {n: synth.normal_bf16((B, H, q_len, D), 9990 + i) for i, n in enumerate("qkv")}
    q8, k8, v8 = (mw.mw_quantize_fp8(to_gpu(inp[n]), sc) for n, sc in (("q", qs), ("k", ks), ("v", vs)))
    o, _ = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, 1, q_len, cache, qs, window=window)
    sync()
    assert ns > 1
    dq = lambda b, sc: oracle.dequantize_fp8(codes(b, sc), sc)
    win = range(len(hist) - window, len(hist))
    win_k = []
    for c in win:
        vals = oracle.dequantize_fp8(codes(hist[c][0], ks), 1.0)
        rot = oracle.rope_rotate(vals, -float(total - at_commit[c]), 0, 44).astype(np.float32)
        win_k.append(oracle.dequantize_fp8(oracle.quantize_fp8(rot, 1.0), ks))
    ro, _ = oracle.cached_chunk_attn(dq(inp["q"], qs), dq(inp["k"], ks), dq(inp["v"], vs), win_k,
                                     [dq(hist[c][1], vs) for c in win], 1, q_len, sink_k=dq(sk, ks),
                                     sink_v=dq(sv, vs))
    assert_close(f"o q_len={q_len} window={window}", to_f64(o), ro, FP8_MAX_ABS, FP8_MEAN_ABS)


def _rotated_window_rollout(mw, L, seed):
    """An e4m3 ring (B1 H2 D128, 5 slots, window 4) whose window chunks carry different pending
    re-shifts (3 per eviction, plus one extra shift of 1 midway), with a 40-token sink."""
    B, H, D, S = 1, 2, 128, 5
    ks, vs = 0.011, 0.012
    cache = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    sk, sv = (mw.mw_quantize_fp8(to_gpu(synth.normal_bf16((B, H, 40, D), seed + i)), sc) for i, sc in ((0, ks), (1, vs)))
    cache.set_sink(sk, sv)
    for t in range(7):
        kb, vb = (synth.normal_bf16((B, H, L, D), seed + 10 + 2 * t + j) for j in range(2))
        if cache.live == S:
            mw.mw_kvcache_evict(cache, 1)
            mw.mw_kvcache_rope_shift(cache, 3, 0, 44)
        if t == 4:
            mw.mw_kvcache_rope_shift(cache, 1, 0, 44)
        mw.mw_kvcache_append(cache, to_gpu(kb), to_gpu(vb))
    return cache, (sk, sv), (B, H, D, S, ks, vs)


def test_fp8_rotation_in_staging_bit_identical_to_separate_pass(mw):
    """e4m3 calls with re-shifts pending and one query tile per head rotate each staged K tile
    inside the attention kernel; calls of more query tiles rotate the window in a separate pass
    into the start of the workspace.  Both run the same arithmetic, so: a 300-row call leaves the
    rotated window in its workspace; a second cache holding those rotated codes in its slots, with nothing pending,
    gives a 64-row call bit for bit the output the shifted cache gives it; and the shifted
    cache's 64-row call (split into key ranges) leaves the workspace's rotated-window bytes
    untouched, i.e. no separate pass ran."""
    import torch
    L, W = 256, 4
    A, (sk, sv), (B, H, D, S, ks, vs) = _rotated_window_rollout(mw, L, seed=9500)
    pend = [A.desc.rope_total - A.desc.rope_at_commit[A.slot_of(c)] for c in range(A.desc.head - W, A.desc.head)]
    assert len(set(pend)) > 1 and max(pend) > 0  # (the newest chunk has nothing pending: identity rotation)
    qs = 0.0105
    kw = W * B * H * L * D
    q2, k2, v2 = (mw.mw_quantize_fp8(to_gpu(synth.normal_bf16((B, H, 300, D), 9560 + i)), qs) for i in range(3))
    ws = torch.full((mw.mw_chunk_attn_cached_workspace_size(A, 1, 300, W),), 0xAB, dtype=torch.uint8, device="cuda")
    mw.mw_chunk_attn_cached_fp8(q2, k2, v2, 1, 300, A, qs, window=W, workspace=ws)
    sync()
    rotated = ws[:kw].view(W, B, H, L, D).clone()
    assert not bool((rotated == 0xAB).all())
    Bc = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    for t in range(W):
        mw.mw_kvcache_append(Bc, to_gpu(synth.normal_bf16((B, H, L, D), 9570 + t)),
                             to_gpu(synth.normal_bf16((B, H, L, D), 9580 + t)))
    for i, c in enumerate(range(A.desc.head - W, A.desc.head)):
        Bc.k_slots[Bc.slot_of(i)].copy_(rotated[i])
        Bc.v_slots[Bc.slot_of(i)].copy_(A.v_slots[A.slot_of(c)])
    Bc.set_sink(sk, sv)
    q8, k8, v8 = (mw.mw_quantize_fp8(to_gpu(synth.normal_bf16((B, H, 64, D), 9590 + i)), qs) for i in range(3))
    ns, _ = mw.mw_chunk_attn_cached_plan(A, 1, 64, W)
    print(f"[case] fp8 rotation in staging vs separate pass, pend={pend}, splits={ns}", flush=True)
    assert ns > 1
    ws_a = torch.full((mw.mw_chunk_attn_cached_workspace_size(A, 1, 64, W),), 0xAB, dtype=torch.uint8, device="cuda")
    oa, la = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, 1, 64, A, qs, window=W, workspace=ws_a, want_lse=True)
    ob, lb = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, 1, 64, Bc, qs, window=W, want_lse=True)
    sync()
    assert bool((ws_a[:kw] == 0xAB).all())
    assert bits_equal(oa, ob)
    assert torch.equal(la, lb)


@pytest.mark.parametrize("L,in_staging", [(32, False), (80, True)])
def test_fp8_rotation_route_vs_oracle(mw, L, in_staging):
    """A 64-row call over a re-shifted window of short chunks.  With 32-token chunks its key range
    spans more window chunks than the kernel's cos/sin tables hold, so the window is rotated in
    the separate pass (the workspace's rotated-window bytes are written); with 80-token chunks it
    rotates in staging, where a 128-key tile spans up to three chunks (the workspace bytes stay
    untouched).  The output against the oracle over the window keys rotated by their pending
    shifts and rounded once, fp8 bar."""
    import torch
    W = 4
    A, (sk, sv), (B, H, D, S, ks, vs) = _rotated_window_rollout(mw, L, seed=9600 + L)
    qs = 0.0105
    kw = W * B * H * L * D
    inp = {n: synth.normal_bf16((B, H, 64, D), 9690 + i) for i, n in enumerate("qkv")}
    q8, k8, v8 = (mw.mw_quantize_fp8(to_gpu(inp[n]), sc) for n, sc in (("q", qs), ("k", ks), ("v", vs)))
    ws = torch.full((mw.mw_chunk_attn_cached_workspace_size(A, 1, 64, W),), 0xAB, dtype=torch.uint8, device="cuda")
    print(f"[case] fp8 rotation route L={L} in_staging={in_staging}", flush=True)
    o, _ = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, 1, 64, A, qs, window=W, workspace=ws)
    sync()
    assert bool((ws[:kw] == 0xAB).all()) == in_staging
    win = list(range(A.desc.head - W, A.desc.head))
    dq = lambda b, sc: oracle.dequantize_fp8(codes(b, sc), sc)
    win_k = []
    for c in win:
        kcodes = u8(A.k_slots[A.slot_of(c)])
        vals = oracle.dequantize_fp8(kcodes, 1.0)
        rot = oracle.rope_rotate(vals, -float(A.desc.rope_total - A.desc.rope_at_commit[A.slot_of(c)]), 0, 44)
        win_k.append(oracle.dequantize_fp8(oracle.quantize_fp8(rot.astype(np.float32), 1.0), ks))
    win_v = [oracle.dequantize_fp8(u8(A.v_slots[A.slot_of(c)]), vs) for c in win]
    ro, _ = oracle.cached_chunk_attn(dq(inp["q"], qs), dq(inp["k"], ks), dq(inp["v"], vs), win_k, win_v, 1, 64,
                                     sink_k=oracle.dequantize_fp8(u8(sk), ks), sink_v=oracle.dequantize_fp8(u8(sv), vs))
    assert_close(f"o L={L}", to_f64(o), ro, FP8_MAX_ABS, FP8_MEAN_ABS)


@pytest.mark.parametrize("L,W,sink_len,nq,qlen,mode", [
    (256, 4, 0, 1, 1, 0),        # one queued row, no sink
    (80, 5, 17, 1, 64, 0),       # 80-token chunks: a 128-key tile spans up to three chunks
    (256, 3, 300, 1, 33, 0),     # a sink longer than two tiles, ragged 33 rows
    (128, 4, 40, 2, 50, 1),      # two queued chunks (100 rows, 128-row configuration), isolated
    (100, 6, 5, 1, 128, 0),      # 128 rows, the whole ring's window after wrapping
    (256, 4, 40, 1, 200, 0),     # 200 rows: the 256-row configuration, one query tile per head
])
def test_fp8_rotation_in_staging_sweep(mw, L, W, sink_len, nq, qlen, mode):
    """Rotation in staging against the separate pass, bit for bit, over shapes that move the
    window's chunk edges, the sink and the ragged end around the staged tiles: the separate pass
    of a 300-row call (two query tiles) on the shifted cache writes the rotated window into its
    workspace; a second
    cache holds those codes with nothing pending; a few-row call gives both caches the same output
    and LSE, and leaves the shifted call's workspace bytes of the rotated window untouched."""
    import torch
    B, H, D = 1, 2, 128
    S = W + 1
    ks, vs, qs = 0.011, 0.012, 0.0105
    seed = 9800 + L + 7 * W + sink_len + qlen
    A = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    sink = None
    if sink_len:
        sink = tuple(mw.mw_quantize_fp8(to_gpu(synth.normal_bf16((B, H, sink_len, D), seed + i)), sc)
                     for i, sc in ((0, ks), (1, vs)))
        A.set_sink(*sink)
    for t in range(W + 3):  # wraps the ring; each eviction re-shifts by 3, one extra shift of 2 midway
        if A.live == S:
            mw.mw_kvcache_evict(A, 1)
            mw.mw_kvcache_rope_shift(A, 3, 0, 44)
        if t == W // 2:
            mw.mw_kvcache_rope_shift(A, 2, 0, 44)
        mw.mw_kvcache_append(A, to_gpu(synth.normal_bf16((B, H, L, D), seed + 10 + 2 * t)),
                             to_gpu(synth.normal_bf16((B, H, L, D), seed + 11 + 2 * t)))
    win = list(range(A.desc.head - W, A.desc.head))
    kw = W * B * H * L * D
    q2 = mw.mw_quantize_fp8(to_gpu(synth.normal_bf16((B, H, 300, D), seed + 50)), qs)
    ws = torch.full((mw.mw_chunk_attn_cached_workspace_size(A, 1, 300, W),), 0xAB, dtype=torch.uint8, device="cuda")
    mw.mw_chunk_attn_cached_fp8(q2, q2, q2, 1, 300, A, qs, window=W, workspace=ws)
    sync()
    rotated = ws[:kw].view(W, B, H, L, D).clone()
    Bc = mw.KVCache(S, B, H, L, D, fp8=True, k_scale=ks, v_scale=vs)
    for t in range(W):
        mw.mw_kvcache_append(Bc, to_gpu(synth.normal_bf16((B, H, L, D), seed + 60 + t)),
                             to_gpu(synth.normal_bf16((B, H, L, D), seed + 70 + t)))
    for i, c in enumerate(win):
        Bc.k_slots[Bc.slot_of(i)].copy_(rotated[i])
        Bc.v_slots[Bc.slot_of(i)].copy_(A.v_slots[A.slot_of(c)])
    if sink:
        Bc.set_sink(*sink)
    q8, k8, v8 = (mw.mw_quantize_fp8(to_gpu(synth.normal_bf16((B, H, nq * qlen, D), seed + 80 + i)), qs)
                  for i in range(3))
    ns, _ = mw.mw_chunk_attn_cached_plan(A, nq, qlen, W, mode)
    print(f"[case] fp8 rotation sweep L={L} W={W} sink={sink_len} nq={nq} qlen={qlen} mode={mode} splits={ns}",
          flush=True)
    ws_a = torch.full((mw.mw_chunk_attn_cached_workspace_size(A, nq, qlen, W),), 0xAB, dtype=torch.uint8,
                      device="cuda")
    oa, la = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, nq, qlen, A, qs, window=W, flags=mode, workspace=ws_a,
                                         want_lse=True)
    ob, lb = mw.mw_chunk_attn_cached_fp8(q8, k8, v8, nq, qlen, Bc, qs, window=W, flags=mode, want_lse=True)
    sync()
    assert bool((ws_a[:kw] == 0xAB).all())
    assert bits_equal(oa, ob)
    assert torch.equal(la, lb)

"""GPU parity of the sink anchor and the RoPE re-shift of the rolling KV cache (paper Sec. 3.5)."""
import numpy as np
import pytest

import oracle
import synth
from helpers import assert_close, bits_equal, f64, to_f64, to_gpu

pytestmark = pytest.mark.gpu


def sync():
    import torch
    torch.cuda.synchronize()


def band(D):
    """Temporal rope band used in these tests: the first D - 4*floor(D/6) dimensions."""
    return 0, D - 4 * (D // 6)


@pytest.mark.parametrize("D", [64, 128])
def test_rope_shift_vs_oracle(mw, D):
    B, H, L, S = 1, 2, 96, 5
    off, cnt = band(D)
    cache = mw.KVCache(S, B, H, L, D)
    chunks = [(synth.normal_bf16((B, H, L, D), 2000 + 2 * i), synth.normal_bf16((B, H, L, D), 2001 + 2 * i))
              for i in range(5)]
    for kc, vc in chunks:
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    mw.mw_kvcache_evict(cache, 2)  # live: chunks 2, 3, 4 in slots 2, 3, 4
    before_k = cache.k_slots.clone()
    before_v = cache.v_slots.clone()
    mw.mw_kvcache_rope_shift(cache, 6, off, cnt, theta=10000.0)
    sync()
    for c in range(5):
        slot = c % S
        got = cache.k_slots[slot]
        if c < 2:  # evicted: untouched
            assert bits_equal(got, before_k[slot])
            continue
        ref = oracle.rope_rotate(f64(chunks[c][0]), -6.0, off, cnt, 10000.0)
        assert_close(f"k chunk {c}", to_f64(got), ref, max_abs=2e-2, mean_abs=2e-3)
        g = to_f64(got)
        assert np.array_equal(g[..., off + cnt:], f64(chunks[c][0])[..., off + cnt:])  # outside the band
    assert bits_equal(cache.v_slots, before_v)  # values are never rotated


def _history(B, H, L, D, n, seed):
    return [(synth.normal_bf16((B, H, L, D), seed + 2 * i), synth.normal_bf16((B, H, L, D), seed + 2 * i + 1))
            for i in range(n)]


@pytest.mark.parametrize("split", [True, False])
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("D,sink_len", [(64, 40), (128, 100)])
def test_cached_attention_with_sink(mw, split, mode, D, sink_len):
    B, H, L, S, nq, qlen, w = 1, 2, 128, 6, 3, 96, 3
    print(f"[case] sink D={D} sink_len={sink_len} mode={mode} split={split}", flush=True)
    cache = mw.KVCache(S, B, H, L, D)
    hist = _history(B, H, L, D, 5, seed=2100 + D)
    for kc, vc in hist:
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    sk, sv = synth.normal_bf16((B, H, sink_len, D), 2200), synth.normal_bf16((B, H, sink_len, D), 2201)
    gk, gv = to_gpu(sk), to_gpu(sv)
    cache.set_sink(gk, gv)
    inp = {n: synth.normal_bf16((B, H, nq * qlen, D), 2300 + i) for i, n in enumerate(("q", "k", "v"))}
    o, lse = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k"]), to_gpu(inp["v"]), nq, qlen, cache, window=w,
                                     flags=mode, want_lse=True, split=split)
    sync()
    ro, rl = oracle.cached_chunk_attn(f64(inp["q"]), f64(inp["k"]), f64(inp["v"]),
                                      [f64(c[0]) for c in hist[-w:]], [f64(c[1]) for c in hist[-w:]], nq, qlen,
                                      mode=mode, sink_k=f64(sk), sink_v=f64(sv))
    assert_close("o", to_f64(o), ro)
    assert_close("lse", to_f64(lse), rl, max_abs=2e-3, mean_abs=2e-4)


def test_sink_mass_probe(mw):
    """V = one-hot(segment): the sink carries softmax mass for every queued row, evicted chunks none."""
    B, H, D, L, S, nq, qlen = 1, 1, 64, 64, 3, 2, 48
    cache = mw.KVCache(S, B, H, L, D)
    for c in range(5):
        if cache.live == 2:
            mw.mw_kvcache_evict(cache, 1)
        vc = np.zeros((B, H, L, D), np.uint16)
        vc[..., 1 + c] = 0x3F80
        mw.mw_kvcache_append(cache, to_gpu(synth.normal_bf16((B, H, L, D), 2400 + c)), to_gpu(vc))
    sv = np.zeros((B, H, 16, D), np.uint16)
    sv[..., 0] = 0x3F80
    gsk, gsv = to_gpu(synth.normal_bf16((B, H, 16, D), 2410)), to_gpu(sv)
    cache.set_sink(gsk, gsv)
    q = to_gpu(synth.normal_bf16((B, H, nq * qlen, D), 2411))
    o, _ = mw.mw_chunk_attn_cached(q, q, to_gpu(np.zeros((B, H, nq * qlen, D), np.uint16)), nq, qlen, cache)
    sync()
    o = to_f64(o)[0, 0]
    assert np.all(o[:, 0] > 0)            # sink
    assert np.all(o[:, 1:4] == 0.0)       # evicted chunks 0, 1, 2
    assert np.all(o[:, 4:6] > 0)          # live chunks 3, 4


def test_rollout_reshift_preserves_relative_positions(mw):
    """Keys carry RoPE at their temporal positions when committed.  Streaming with FIFO
    eviction and re-shifting of the retained keys by the evicted positions, with queries at
    re-indexed positions, gives the same attention as absolute positions without any re-shift
    (relative positions inside the window are unchanged), within the parity bar.  The sink keeps
    its first position and is never shifted, so relative to the window it behaves as if it sat
    at absolute position = total shift: the reference places it there."""
    B, H, D, L, S, W, nq, frames = 1, 2, 128, 64, 4, 3, 2, 2  # 2 positions (frames) per chunk, 32 tokens each
    off, cnt = band(D)
    tok_pos = lambda start: np.repeat(np.arange(start, start + frames), L // frames).astype(float)
    sink_len = L // frames  # one frame
    raw_sink = [synth.normal_bf16((B, H, sink_len, D), 2500 + i) for i in range(2)]
    sink_k = synth.f32_to_bf16_bits(oracle.rope_rotate(f64(raw_sink[0]), np.zeros(sink_len), off, cnt).astype(np.float32))
    cache = mw.KVCache(S, B, H, L, D)
    gsk, gsv = to_gpu(sink_k), to_gpu(raw_sink[1])
    cache.set_sink(gsk, gsv)
    committed = {}  # chunk id -> (k with RoPE at absolute positions, v), fp64
    shift_total = 0
    for t in range(7):
        p0 = 1 + t * frames  # chunk t covers frames 1 + t*frames ... (frame 0 is the sink)
        kraw = synth.normal_bf16((B, H, L, D), 2600 + 3 * t)
        v = synth.normal_bf16((B, H, L, D), 2601 + 3 * t)
        k_abs = oracle.rope_rotate(f64(kraw), tok_pos(p0), off, cnt)
        # the committed key is RoPE'd at its position in the current (re-indexed) frame
        k_cur = synth.f32_to_bf16_bits(oracle.rope_rotate(f64(kraw), tok_pos(p0 - shift_total), off, cnt).astype(np.float32))
        committed[t] = (synth.bf16_bits_to_f64(synth.f32_to_bf16_bits(k_abs.astype(np.float32))), f64(v))
        mw.mw_kvcache_append(cache, to_gpu(k_cur), to_gpu(v))
        if cache.live > W:
            n = cache.live - W
            mw.mw_kvcache_evict(cache, n)
            mw.mw_kvcache_rope_shift(cache, n * frames, off, cnt)  # re-index after evicting n chunks
            shift_total += n * frames
        if t < 3:
            continue
        # two queued chunks at the next positions, RoPE'd in the current frame
        qp0 = 1 + (t + 1) * frames
        qraw = synth.normal_bf16((B, H, nq * L, D), 2700 + t)
        knr = synth.normal_bf16((B, H, nq * L, D), 2710 + t)
        vn = synth.normal_bf16((B, H, nq * L, D), 2720 + t)
        qpos = np.concatenate([tok_pos(qp0 + j * frames) for j in range(nq)])
        rot = lambda x, pos: synth.f32_to_bf16_bits(oracle.rope_rotate(f64(x), pos, off, cnt).astype(np.float32))
        o, _ = mw.mw_chunk_attn_cached(to_gpu(rot(qraw, qpos - shift_total)), to_gpu(rot(knr, qpos - shift_total)),
                                       to_gpu(vn), nq, L, cache)
        sync()
        live = list(range(t + 1 - cache.live, t + 1))
        ro, _ = oracle.cached_chunk_attn(oracle.rope_rotate(f64(qraw), qpos, off, cnt),
                                         oracle.rope_rotate(f64(knr), qpos, off, cnt), f64(vn),
                                         [committed[c][0] for c in live], [committed[c][1] for c in live], nq, L,
                                         sink_k=oracle.rope_rotate(f64(raw_sink[0]), np.full(sink_len, float(shift_total)),
                                                                   off, cnt),
                                         sink_v=f64(raw_sink[1]))
        assert_close(f"step {t} (shift {shift_total})", to_f64(o), ro)


def test_rope_reshift_drift_over_cache_life(mw):
    """A key's whole life in the paper's largest cache (24 chunks): it is re-shifted once per
    eviction, so up to 24 times, and each in-place shift rounds it to bf16 again.  Every key
    after 24 shifts of 3 positions is compared with one fp64 rotation of the committed key by
    the summed 72 positions.  Bound: each shift adds a rounding error of at most u = 2^-8
    (bf16's unit roundoff) relative to each rotated element, and a rotation keeps the norm of a
    pair, so after n shifts a pair's error is at most n * sqrt(2) * u * (1 + n u) times its norm
    (plus fp32 rotation error, far smaller).  The drift must also leave the attention of two
    queued chunks over the drifted window within the parity bar of the exact rotation."""
    B, H, L, D, W, n, step = 1, 2, 128, 128, 24, 24, 3
    off, cnt = band(D)
    print(f"[case] rope drift: {n} shifts of {step} over a {W}-chunk window, D={D}", flush=True)
    cache = mw.KVCache(W + 1, B, H, L, D)
    chunks = _history(B, H, L, D, W, 2800)
    for kc, vc in chunks:
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    for _ in range(n):
        mw.mw_kvcache_rope_shift(cache, step, off, cnt)
    sync()
    u = 2.0 ** -8
    worst_ratio, errs = 0.0, []
    exact = []
    for c in range(W):
        k0 = f64(chunks[c][0])
        ref = oracle.rope_rotate(k0, -float(n * step), off, cnt)
        exact.append(ref)
        got = to_f64(cache.k_slots[cache.slot_of(c)])
        assert np.array_equal(got[..., off + cnt:], k0[..., off + cnt:])  # outside the band: never touched
        e = np.abs(got - ref)[..., off:off + cnt]
        pair_norm = np.sqrt(k0[..., off:off + cnt:2] ** 2 + k0[..., off + 1:off + cnt:2] ** 2)
        bound = n * np.sqrt(2.0) * u * (1.0 + n * u) * np.repeat(pair_norm, 2, axis=-1) + 1e-6
        worst_ratio = max(worst_ratio, float((e / bound).max()))
        errs.append(e)
    e = np.concatenate([x.ravel() for x in errs])
    print(f"[drift] after {n} shifts: max_abs={e.max():.3e} mean_abs={e.mean():.3e} rms={np.sqrt((e ** 2).mean()):.3e} "
          f"worst fraction of the bound={worst_ratio:.3f}", flush=True)
    assert worst_ratio <= 1.0
    # attention over the drifted window vs the exact single rotation
    nq = 2
    inp = {x: synth.normal_bf16((B, H, nq * L, D), 2990 + i) for i, x in enumerate("qkv")}
    o, _ = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k"]), to_gpu(inp["v"]), nq, L, cache, window=W)
    sync()
    ro, _ = oracle.cached_chunk_attn(f64(inp["q"]), f64(inp["k"]), f64(inp["v"]), exact,
                                     [f64(cv) for _, cv in chunks], nq, L)
    assert_close("attention over the drifted window", to_f64(o), ro)

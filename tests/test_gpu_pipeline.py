"""A streaming rollout driven by the library's plan of the pipelined denoiser (paper Sec. 3.5):
each tick runs cached attention of the in-flight chunks over [sink | cache], then commits the
chunks that reached tau = 0, evicts and re-shifts as planned.  Queries and keys carry RoPE at
their positions in the re-indexed sequence the plan gives; the attention must equal the
oracle's with every token at its absolute position (the sink, never shifted, sitting the total
shift further along), within the parity bar, at every tick."""
import numpy as np
import pytest

import oracle
import synth
from helpers import assert_close, f64, to_f64, to_gpu

pytestmark = pytest.mark.gpu


def rot_bits(x, pos, off, cnt):
    return synth.f32_to_bf16_bits(oracle.rope_rotate(f64(x), pos, off, cnt).astype(np.float32))


@pytest.mark.parametrize("D,window,stride,cache_chunks", [(64, 4, 1, 3), (128, 6, 2, 4)])
def test_plan_driven_rollout(mw, D, window, stride, cache_chunks):
    import torch
    B, H, f, tpf, sink_frames, N = 1, 2, 2, 16, 1, 9     # 2 frames of 16 tokens per chunk
    L = f * tpf
    off, cnt = 0, D - 4 * (D // 6)
    cfg = mw.sched_config(window, stride, N, cache_chunks, f, sink_frames=sink_frames, shift=3.0)
    ticks = mw.mw_sched_num_ticks(cfg)
    print(f"[case] plan-driven rollout D={D} W={window} r={stride} C={cache_chunks} ticks={ticks}", flush=True)
    cache = mw.KVCache(cache_chunks + stride, B, H, L, D)
    tok_frames = lambda f0: np.repeat(np.arange(f0, f0 + f), tpf).astype(float)
    sink_raw = [synth.normal_bf16((B, H, sink_frames * tpf, D), 6000 + i) for i in range(2)]
    sink_pos = np.repeat(np.arange(sink_frames), tpf).astype(float)
    gsk, gsv = to_gpu(rot_bits(sink_raw[0], sink_pos, off, cnt)), to_gpu(sink_raw[1])
    cache.set_sink(gsk, gsv)
    raw = lambda c, k, w: synth.normal_bf16((B, H, L, D), 7000 + 1000 * w + 10 * c + k)  # chunk c, update k
    committed = {}          # chunk -> (k at its absolute frames, v) in fp64
    cached = []             # chunk ids in the cache, oldest first
    shift_total = 0
    for t in range(ticks):
        p = mw.mw_sched_plan(cfg, t)
        assert p["pos_first"] == sink_frames + len(cached) * f
        n, ids = p["n_active"], p["ids"]
        U = p["updates_per_chunk"]
        ks = [t - c // stride for c in ids]                   # updates each in-flight chunk has had
        q_raw = [raw(c, k, 0) for c, k in zip(ids, ks)]
        k_raw = [raw(c, k, 1) for c, k in zip(ids, ks)]
        v_new = np.concatenate([raw(c, k, 2) for c, k in zip(ids, ks)], axis=2)
        cur = [tok_frames(p["pos_first"] + a * f) for a in range(n)]                 # re-indexed frames
        absf = [tok_frames(sink_frames + c * f) for c in ids]                        # absolute frames
        q_cur = np.concatenate([rot_bits(x, pos, off, cnt) for x, pos in zip(q_raw, cur)], axis=2)
        k_cur = np.concatenate([rot_bits(x, pos, off, cnt) for x, pos in zip(k_raw, cur)], axis=2)
        o, _ = mw.mw_chunk_attn_cached(to_gpu(q_cur), to_gpu(k_cur), to_gpu(v_new), n, L, cache)
        torch.cuda.synchronize()
        q_abs = np.concatenate([oracle.rope_rotate(f64(x), pos, off, cnt) for x, pos in zip(q_raw, absf)], axis=2)
        k_abs = np.concatenate([oracle.rope_rotate(f64(x), pos, off, cnt) for x, pos in zip(k_raw, absf)], axis=2)
        ro, _ = oracle.cached_chunk_attn(q_abs, k_abs, f64(v_new), [committed[c][0] for c in cached],
                                         [committed[c][1] for c in cached], n, L,
                                         sink_k=oracle.rope_rotate(f64(sink_raw[0]), sink_pos + shift_total, off, cnt),
                                         sink_v=f64(sink_raw[1]))
        assert_close(f"tick {t} (in flight {ids[0]}..{ids[-1]}, shift {shift_total})", to_f64(o), ro)
        # commit the chunks that reached tau = 0: their keys and values of the last update
        for a, c in enumerate(p["committed"]):
            assert ks[a] == U - 1
            kb = k_cur[:, :, a * L:(a + 1) * L]
            vb = v_new[:, :, a * L:(a + 1) * L]
            mw.mw_kvcache_append(cache, to_gpu(np.ascontiguousarray(kb)), to_gpu(np.ascontiguousarray(vb)))
            committed[c] = (oracle.rope_rotate(f64(k_raw[a]), absf[a], off, cnt), f64(vb))
            cached.append(c)
        if p["n_evict"]:
            mw.mw_kvcache_evict(cache, p["n_evict"])
            mw.mw_kvcache_rope_shift(cache, p["rope_shift"], off, cnt)
            del cached[:p["n_evict"]]
            shift_total += p["rope_shift"]
        assert cache.live == p["cache_live"] == len(cached)

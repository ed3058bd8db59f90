"""GPU parity of the rolling KV cache and cached chunk attention (paper Sec. 3.5)."""
import numpy as np
import pytest

import oracle
import synth
from helpers import assert_close, bits_equal, f64, to_f64, to_gpu

pytestmark = pytest.mark.gpu


def sync():
    import torch
    torch.cuda.synchronize()


def make_chunks(n, B, H, L, D, seed):
    return [(synth.normal_bf16((B, H, L, D), seed + 2 * i), synth.normal_bf16((B, H, L, D), seed + 2 * i + 1))
            for i in range(n)]


def queued(B, H, nq, qlen, D, seed):
    return {n: synth.normal_bf16((B, H, nq * qlen, D), seed + i) for i, n in enumerate(("q", "k_new", "v_new"))}


@pytest.mark.parametrize("split", [True, False])
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("B,H,D,L,S,n_commit,window,nq,qlen", [
    (1, 2, 64, 96, 4, 6, 3, 2, 96),      # wrapped ring, chunk edges inside tiles
    (2, 1, 128, 160, 5, 5, -1, 3, 160),  # all live chunks
    (1, 2, 64, 100, 3, 2, 0, 2, 70),     # empty window, queued chunks of another length
    (1, 1, 128, 64, 8, 9, 7, 4, 33),     # short queued chunks
    (1, 2, 72, 150, 4, 6, 3, 3, 150),    # D=72 (the 0.5B model's head width)
    (2, 4, 64, 96, 4, 6, 3, 2, 96),      # B*H = 8: the split-major work order with XCD-aware heads
    (1, 8, 128, 160, 5, 5, -1, 3, 160),
])
def test_cached_attention_vs_oracle(mw, split, mode, B, H, D, L, S, n_commit, window, nq, qlen):
    print(f"[case] cached split={split} mode={mode} B={B} H={H} D={D} L={L} S={S} commits={n_commit} w={window} "
          f"nq={nq} qlen={qlen}", flush=True)
    cache = mw.KVCache(S, B, H, L, D)
    chunks = make_chunks(n_commit, B, H, L, D, seed=300 + L)
    ring = oracle.RingModel(S)
    for kc, vc in chunks:
        if ring.live == S:
            ring.evict(1)
            mw.mw_kvcache_evict(cache, 1)
        slot = mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
        assert slot == ring.append()
    win = ring.window(None if window == -1 else window)
    inp = queued(B, H, nq, qlen, D, seed=400 + qlen)
    o, lse = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(inp["v_new"]), nq, qlen, cache,
                                     window=window, flags=mode, want_lse=True, split=split)
    sync()
    ro, rl = oracle.cached_chunk_attn(f64(inp["q"]), f64(inp["k_new"]), f64(inp["v_new"]),
                                      [f64(chunks[c][0]) for c in win], [f64(chunks[c][1]) for c in win],
                                      nq, qlen, mode=mode)
    assert_close("o", to_f64(o), ro)
    assert_close("lse", to_f64(lse), rl, max_abs=2e-3, mean_abs=2e-4)


def test_cached_full_history_equals_training_rows(mw):
    """A window holding all committed history gives the training forward's rows (bit-exact:
    both visit the same keys in the same order)."""
    import torch
    B, H, D, L, nq = 1, 2, 128, 192, 3
    hist = make_chunks(4, B, H, L, D, seed=500)
    cache = mw.KVCache(6, B, H, L, D)
    for kc, vc in hist:
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    inp = queued(B, H, nq, L, D, seed=600)
    # single pass: the split path sums partial results in another order
    o, lse = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(inp["v_new"]), nq, L, cache,
                                     want_lse=True, split=False)
    K = np.concatenate([c[0] for c in hist] + [inp["k_new"]], axis=2)
    V = np.concatenate([c[1] for c in hist] + [inp["v_new"]], axis=2)
    Q = np.concatenate([np.zeros_like(c[0]) for c in hist] + [inp["q"]], axis=2)
    of, lf = mw.mw_block_causal_attn_fwd(to_gpu(Q), to_gpu(K), to_gpu(V), L)
    sync()
    n0 = len(hist) * L
    assert bits_equal(o, of[:, :, n0:].contiguous())
    assert torch.equal(lse, lf[:, :, n0:].contiguous())


@pytest.mark.parametrize("split", [True, False])
def test_wraparound_invariance(mw, split):
    """The same logical window at different ring offsets gives bit-identical outputs
    (split boundaries depend only on the shape, so this holds with splitting too)."""
    B, H, D, L, S, w, nq = 1, 2, 64, 128, 5, 3, 2
    chunks = make_chunks(w, B, H, L, D, seed=700)
    inp = queued(B, H, nq, L, D, seed=800)
    filler = make_chunks(1, B, H, L, D, seed=900)[0]
    outs = []
    for offset in range(S):
        cache = mw.KVCache(S, B, H, L, D)
        for _ in range(offset):  # advance the ring by committing and evicting filler chunks
            mw.mw_kvcache_append(cache, to_gpu(filler[0]), to_gpu(filler[1]))
            mw.mw_kvcache_evict(cache, 1)
        for kc, vc in chunks:
            mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
        assert cache.slot_of(cache.head - w) == offset % S
        o, _ = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(inp["v_new"]), nq, L, cache,
                                       split=split)
        sync()
        outs.append(o)
    for o in outs[1:]:
        assert bits_equal(o, outs[0])


def test_cached_mass_probe_no_mass_on_evicted(mw):
    """V = one-hot(logical chunk id): exactly zero mass on evicted chunks and on later queued chunks."""
    B, H, D, L, S, nq, qlen = 1, 1, 64, 80, 4, 3, 50
    cache = mw.KVCache(S, B, H, L, D)
    ring = oracle.RingModel(S)
    ids_in_slot = {}
    for c in range(7):  # commit 7 chunks, keep 3 live
        if ring.live == 3:
            ring.evict(1)
            mw.mw_kvcache_evict(cache, 1)
        kc = synth.normal_bf16((B, H, L, D), 1000 + c)
        vc = np.zeros((B, H, L, D), np.uint16)
        vc[..., c] = 0x3F80
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
        ring.append()
    inp = queued(B, H, nq, qlen, D, seed=1100)
    vn = np.zeros((B, H, nq * qlen, D), np.uint16)
    for j in range(nq):
        vn[:, :, j * qlen:(j + 1) * qlen, 7 + j] = 0x3F80
    for mode in (0, 1):
        o, _ = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(vn), nq, qlen, cache, flags=mode)
        sync()
        o = to_f64(o)
        assert np.all(o[..., 0:4] == 0.0)  # chunks 0..3 were evicted
        for j in range(nq):
            rows = o[0, 0, j * qlen:(j + 1) * qlen]
            assert np.all(rows[:, 7 + j + 1:7 + nq] == 0.0)
            if mode == 1:
                assert np.all(rows[:, 7:7 + j] == 0.0)
            assert np.all(rows[:, 4:7].sum(axis=1) > 0)
        assert np.max(np.abs(o.sum(axis=-1) - 1.0)) < 2e-2


def test_ring_errors_and_slots(mw):
    import torch
    B, H, D, L, S = 1, 1, 64, 16, 3
    cache = mw.KVCache(S, B, H, L, D)
    chunks = make_chunks(4, B, H, L, D, seed=1200)
    for i in range(3):
        mw.mw_kvcache_append(cache, to_gpu(chunks[i][0]), to_gpu(chunks[i][1]))
    with pytest.raises(mw.MWError) as e:
        mw.mw_kvcache_append(cache, to_gpu(chunks[3][0]), to_gpu(chunks[3][1]))
    assert e.value.code == mw.MW_EFULL
    with pytest.raises(mw.MWError) as e:
        mw.mw_kvcache_evict(cache, 4)
    assert e.value.code == mw.MW_EEMPTY
    q = to_gpu(synth.normal_bf16((B, H, L, D), 1))
    with pytest.raises(mw.MWError) as e:
        mw.mw_chunk_attn_cached(q, q, q, 1, L, cache, window=4)
    assert e.value.code == mw.MW_EINVAL
    mw.mw_kvcache_evict(cache, 1)
    mw.mw_kvcache_append(cache, to_gpu(chunks[3][0]), to_gpu(chunks[3][1]))
    sync()
    for c in range(1, 4):
        slot = cache.slot_of(c)
        assert slot == c % S
        assert bits_equal(cache.k_slots[slot], to_gpu(chunks[c][0]))
        assert bits_equal(cache.v_slots[slot], to_gpu(chunks[c][1]))
    assert cache.slot_of(0) == -1


def test_cached_rejects_bad_lse(mw):
    """A caller-supplied lse of the wrong dtype, shape or layout raises before any launch, for
    the bf16 and the e4m3 cached calls (the kernels write fp32 at [b, h, row])."""
    import torch
    B, H, D, L, S, nq = 1, 2, 128, 32, 3, 2
    q = to_gpu(synth.normal_bf16((B, H, nq * L, D), 5))
    q8 = mw.mw_quantize_fp8(q, 0.01)
    bad = [torch.empty((B, H, nq * L), dtype=torch.bfloat16, device="cuda"),
           torch.empty((B, H), dtype=torch.float32, device="cuda"),
           torch.empty((B, H, nq * L - 1), dtype=torch.float32, device="cuda"),
           torch.empty((B, nq * L, H), dtype=torch.float32, device="cuda").transpose(1, 2)]
    for fp8 in (False, True):
        cache = mw.KVCache(S, B, H, L, D, fp8=fp8, k_scale=0.01, v_scale=0.01)
        mw.mw_kvcache_append(cache, q[:, :, :L], q[:, :, :L])
        for lse in bad:
            with pytest.raises(ValueError):
                if fp8:
                    mw.mw_chunk_attn_cached_fp8(q8, q8, q8, nq, L, cache, 0.01, lse=lse)
                else:
                    mw.mw_chunk_attn_cached(q, q, q, nq, L, cache, lse=lse)
    sync()


def test_host_workspace_rejected(mw):
    """A workspace in host memory raises before any launch (the kernels would write their
    partials through it), for the bf16 and e4m3 cached calls and the training backward."""
    import torch
    B, H, D, L, S, nq = 1, 2, 128, 64, 3, 1
    q = to_gpu(synth.normal_bf16((B, H, nq * L, D), 6))
    q8 = mw.mw_quantize_fp8(q, 0.01)
    host_ws = torch.empty(1 << 22, dtype=torch.uint8)
    for fp8 in (False, True):
        cache = mw.KVCache(S, B, H, L, D, fp8=fp8, k_scale=0.01, v_scale=0.01)
        mw.mw_kvcache_append(cache, q, q)
        with pytest.raises(ValueError):
            if fp8:
                mw.mw_chunk_attn_cached_fp8(q8, q8, q8, nq, L, cache, 0.01, workspace=host_ws)
            else:
                mw.mw_chunk_attn_cached(q, q, q, nq, L, cache, workspace=host_ws)
    o, lse = mw.mw_block_causal_attn_fwd(q, q, q, L)
    with pytest.raises(ValueError):
        mw.mw_block_causal_attn_bwd(q, q, q, o, o, lse, L, workspace=host_ws)
    sync()


@pytest.mark.parametrize("q_len", [64, 128, 256, 300, 512])
def test_decode_shape_split_vs_oracle(mw, q_len):
    """One short queued chunk over a full 6-chunk window (B1 H16 D128, 2640-token chunks):
    few query tiles, so the key range is split over many workgroups."""
    s = synth.STREAM
    print(f"[case] decode q_len={q_len}", flush=True)
    cache = mw.KVCache(s.slots, s.B, s.H, s.chunk_len, s.D)
    hist = make_chunks(s.window, s.B, s.H, s.chunk_len, s.D, seed=s.seed_base + 70)
    for kc, vc in hist:
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    assert mw.mw_chunk_attn_cached_workspace_size(cache, 1, q_len) > 0
    inp = queued(s.B, s.H, 1, q_len, s.D, seed=s.seed_base + 80 + q_len)
    o, lse = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(inp["v_new"]), 1, q_len, cache,
                                     want_lse=True)
    o1, _ = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(inp["v_new"]), 1, q_len, cache,
                                    split=False)
    sync()
    ro, rl = oracle.cached_chunk_attn(f64(inp["q"]), f64(inp["k_new"]), f64(inp["v_new"]),
                                      [f64(c[0]) for c in hist], [f64(c[1]) for c in hist], 1, q_len)
    assert_close("o split", to_f64(o), ro)
    assert_close("lse split", to_f64(lse), rl, max_abs=2e-3, mean_abs=2e-4)
    assert_close("o single pass", to_f64(o1), ro)


@pytest.mark.parametrize("split", [True, False])
@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("B,H,L,S,n_commit,window,nq,qlen,sink_len", [
    (1, 2, 250, 4, 5, 3, 1, 64, 0),     # 64 rows: two key groups of two row waves, 64-key tiles four deep
    (1, 2, 600, 4, 5, 3, 2, 30, 40),    # 60 rows in two queued chunks, sink: key ranges cross sink/window/queued
    (1, 3, 300, 4, 6, 3, 2, 50, 0),     # 100 rows in two queued chunks: two key groups of four
    (2, 1, 200, 5, 5, 4, 3, 40, 17),    # 120 rows, three queued chunks, sink of 17 tokens
    (1, 1, 96, 3, 4, 2, 1, 7, 0),       # 7 rows over 199 keys: fewer tiles than the pipeline holds, ragged end
    (1, 2, 130, 4, 6, -1, 2, 33, 5),    # all live chunks, ragged 66 rows, sink
    (1, 2, 200, 4, 5, 3, 3, 100, 9),    # 300 rows: three 128-row tiles of two key groups, sink
])
def test_few_rows_key_groups_vs_oracle(mw, split, mode, B, H, L, S, n_commit, window, nq, qlen, sink_len):
    """Cached attention with at most 128 queued rows (D=128), the configuration whose waves
    split the keys of each step into groups and merge at the end; both visibility modes, with
    and without the key-range split, sinks and ragged row counts."""
    D = 128
    print(f"[case] few rows split={split} mode={mode} B={B} H={H} L={L} S={S} commits={n_commit} w={window} "
          f"nq={nq} qlen={qlen} sink={sink_len}", flush=True)
    cache = mw.KVCache(S, B, H, L, D)
    chunks = make_chunks(n_commit, B, H, L, D, seed=3100 + L)
    ring = oracle.RingModel(S)
    for kc, vc in chunks:
        if ring.live == S:
            ring.evict(1)
            mw.mw_kvcache_evict(cache, 1)
        assert mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc)) == ring.append()
    sk = sv = None
    if sink_len:
        sk, sv = (synth.normal_bf16((B, H, sink_len, D), 3200 + i) for i in range(2))
        gsk, gsv = to_gpu(sk), to_gpu(sv)
        cache.set_sink(gsk, gsv)
    win = ring.window(None if window == -1 else window)
    inp = queued(B, H, nq, qlen, D, seed=3300 + qlen)
    o, lse = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(inp["v_new"]), nq, qlen, cache,
                                     window=window, flags=mode, want_lse=True, split=split)
    sync()
    ro, rl = oracle.cached_chunk_attn(f64(inp["q"]), f64(inp["k_new"]), f64(inp["v_new"]),
                                      [f64(chunks[c][0]) for c in win], [f64(chunks[c][1]) for c in win],
                                      nq, qlen, mode=mode,
                                      sink_k=None if sk is None else f64(sk), sink_v=None if sv is None else f64(sv))
    assert_close("o", to_f64(o), ro)
    assert_close("lse", to_f64(lse), rl, max_abs=2e-3, mean_abs=2e-4)


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("H,D,window", [(8, 128, 2), (16, 64, 1)])
def test_hybrid_split_plan_vs_oracle(mw, mode, H, D, window):
    """Three 1500-token chunks over a 2-chunk (B1 H8 D128) or 1-chunk (B1 H16 D64, two row blocks
    per wave) window.  Isolated, the split plan keeps the 6 heaviest of each head's 18 query tiles
    whole and splits the others over 2 key ranges (whole tiles write O directly, the merge covers
    only the split rows); queued-causal splits every tile.  Both against the oracle and against
    the unsplit pass."""
    B, L, nq = 1, 1500, 3
    S = window + 2
    print(f"[case] hybrid split plan mode={mode} B={B} H={H} D={D} L={L} nq={nq} w={window}", flush=True)
    cache = mw.KVCache(S, B, H, L, D)
    chunks = make_chunks(window, B, H, L, D, seed=5100 + D)
    for kc, vc in chunks:
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    ns, nw = mw.mw_chunk_attn_cached_plan(cache, nq, L, window, mode)
    assert (ns, nw) == ((2, 6) if mode == 1 else (2, 0))
    inp = queued(B, H, nq, L, D, seed=5200 + D)
    args = (to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(inp["v_new"]), nq, L, cache)
    o, lse = mw.mw_chunk_attn_cached(*args, window=window, flags=mode, want_lse=True)
    o1, lse1 = mw.mw_chunk_attn_cached(*args, window=window, flags=mode, want_lse=True, split=False)
    sync()
    ro, rl = oracle.cached_chunk_attn(f64(inp["q"]), f64(inp["k_new"]), f64(inp["v_new"]),
                                      [f64(c[0]) for c in chunks], [f64(c[1]) for c in chunks], nq, L, mode=mode)
    assert_close("o", to_f64(o), ro)
    assert_close("lse", to_f64(lse), rl, max_abs=2e-3, mean_abs=2e-4)
    # the whole tiles (rows past the split rows) run the unsplit pass's arithmetic
    rows = (18 - nw) * 256 if ns > 1 else 0
    assert np.array_equal(to_f64(o)[:, :, rows:], to_f64(o1)[:, :, rows:])
    assert np.array_equal(to_f64(lse)[:, :, rows:], to_f64(lse1)[:, :, rows:])


@pytest.fixture(scope="module")
def stream_run(mw):
    s = synth.STREAM
    print(f"[case] {s.name}", flush=True)
    cache = mw.KVCache(s.slots, s.B, s.H, s.chunk_len, s.D)
    hist = make_chunks(s.slots, s.B, s.H, s.chunk_len, s.D, seed=s.seed_base + 50)
    for kc, vc in hist:  # 8 commits, then keep the newest 6
        mw.mw_kvcache_append(cache, to_gpu(kc), to_gpu(vc))
    mw.mw_kvcache_evict(cache, s.slots - s.window)
    inp = synth.stream_step_inputs(s, 0, which=("q", "k_new", "v_new"))
    out = {}
    for mode in (0, 1):
        o, lse = mw.mw_chunk_attn_cached(to_gpu(inp["q"]), to_gpu(inp["k_new"]), to_gpu(inp["v_new"]), s.n_queued,
                                         s.q_len, cache, window=s.window, flags=mode, want_lse=True)
        out[mode] = (to_f64(o), to_f64(lse))
    sync()
    return s, hist[-s.window:], inp, out


@pytest.mark.parametrize("mode", [0, 1])
def test_stream_config_all_heads(stream_run, mode):
    """4 in-flight chunks of 2640 tokens over a 6-chunk window in an 8-slot ring, every head."""
    s, win, inp, out = stream_run
    ro, rl = oracle.cached_chunk_attn(f64(inp["q"]), f64(inp["k_new"]), f64(inp["v_new"]),
                                      [f64(c[0]) for c in win], [f64(c[1]) for c in win], s.n_queued, s.q_len,
                                      mode=mode)
    assert_close(f"o mode{mode}", out[mode][0], ro)
    assert_close(f"lse mode{mode}", out[mode][1], rl, max_abs=2e-3, mean_abs=2e-4)


def test_rollout_200_steps(mw):
    """200 chunk steps: commit, evict to the window, cached attention.  Slot indexing and slot
    contents are bit-exact against the integer ring model every step; attention output is checked
    against the oracle on two heads at steps 0-7, 50, 100 and 199."""
    import torch
    s = synth.ROLLOUT
    print(f"[case] {s.name}", flush=True)
    cache = mw.KVCache(s.slots, s.B, s.H, s.chunk_len, s.D)
    ring = oracle.RingModel(s.slots)
    check_steps = set(range(8)) | {50, 100, 199}
    heads = [(0, 0), (0, s.H - 1)]
    committed = {}  # logical chunk -> (k bits, v bits) for the live window
    fixed = None
    for t in range(s.steps):
        cbits = synth.stream_step_inputs(s, t, which=("k_commit", "v_commit"))
        kc, vc = to_gpu(cbits["k_commit"]), to_gpu(cbits["v_commit"])
        slot = mw.mw_kvcache_append(cache, kc, vc)
        assert slot == ring.append() == t % s.slots
        committed[t] = (cbits["k_commit"], cbits["v_commit"])
        if ring.live > s.window:
            n = ring.live - s.window
            ring.evict(n)
            mw.mw_kvcache_evict(cache, n)
        for c in range(max(0, t - s.slots - 1), t + 1):
            assert cache.slot_of(c) == ring.slot_of(c)
        for c in list(committed):
            if c < ring.tail:
                del committed[c]
        if t in check_steps:
            qb = synth.stream_step_inputs(s, t, which=("q", "k_new", "v_new"))
            q, kn, vn = (to_gpu(qb[n]) for n in ("q", "k_new", "v_new"))
        else:
            if fixed is None:
                fixed = tuple(to_gpu(b) for b in synth.stream_step_inputs(s, 1, which=("q", "k_new", "v_new")).values())
            q, kn, vn = fixed
        o, _ = mw.mw_chunk_attn_cached(q, kn, vn, s.n_queued, s.q_len, cache, window=-1)
        torch.cuda.synchronize()
        assert bits_equal(cache.k_slots[slot], kc) and bits_equal(cache.v_slots[slot], vc)
        if t in check_steps:
            print(f"[step] {t}: window {ring.window()}", flush=True)
            win = ring.window()
            ro, _ = oracle.cached_chunk_attn(f64(qb["q"]), f64(qb["k_new"]), f64(qb["v_new"]),
                                             [f64(committed[c][0]) for c in win], [f64(committed[c][1]) for c in win],
                                             s.n_queued, s.q_len, heads=heads)
            go = to_f64(o)
            for b, h in heads:
                assert_close(f"step {t} o h{h}", go[b, h], ro[b, h])
            # every live chunk still holds exactly what was committed
            for c in win:
                sl = cache.slot_of(c)
                assert bits_equal(cache.k_slots[sl], to_gpu(committed[c][0]))


def test_snapshot_restore_continue_bit_identical(mw):
    """Checkpoint and resume of a rollout: after k steps the ring descriptor (KVCache.snapshot)
    and the slot buffers are saved; the rollout continues n steps (commit, evict to the window,
    cached attention, RoPE re-shift); then the saved state is restored and the same n steps run
    again.  Every output, every slot and the ring counters match the first continuation
    bit for bit; the slot numbering agrees with the ring model throughout."""
    import torch
    B, H, L, D, S, W, nq, k, n = 1, 2, 96, 128, 5, 3, 2, 7, 6
    cache = mw.KVCache(S, B, H, L, D)
    ring = oracle.RingModel(S)

    def step(t):
        kc, vc = (to_gpu(synth.normal_bf16((B, H, L, D), 3000 + 2 * t + j)) for j in range(2))
        slot = mw.mw_kvcache_append(cache, kc, vc)
        if cache.live > W:
            mw.mw_kvcache_evict(cache, cache.live - W)
            mw.mw_kvcache_rope_shift(cache, 2, 0, 44)
        q, kn, vn = (to_gpu(synth.normal_bf16((B, H, nq * L, D), 3500 + 3 * t + j)) for j in range(3))
        o, lse = mw.mw_chunk_attn_cached(q, kn, vn, nq, L, cache, window=cache.live, want_lse=True)
        return slot, o, lse

    for t in range(k):
        slot, _, _ = step(t)
        assert slot == ring.append()
        if ring.live > W:
            ring.evict(ring.live - W)
    snap = cache.snapshot()
    saved_k, saved_v = cache.k_slots.clone(), cache.v_slots.clone()
    first = []
    for t in range(k, k + n):
        first.append(step(t))
    sync()
    end_state = (cache.snapshot(), cache.k_slots.clone(), cache.v_slots.clone())
    # restore and run the same steps again
    cache.restore(snap)
    cache.k_slots.copy_(saved_k)
    cache.v_slots.copy_(saved_v)
    for i, t in enumerate(range(k, k + n)):
        slot, o, lse = step(t)
        assert slot == first[i][0] == ring.append()
        if ring.live > W:
            ring.evict(ring.live - W)
        assert bits_equal(o, first[i][1]), f"output of step {t} differs after restore"
        assert torch.equal(lse, first[i][2])
    sync()
    assert cache.snapshot() == end_state[0]
    assert bits_equal(cache.k_slots, end_state[1]) and bits_equal(cache.v_slots, end_state[2])

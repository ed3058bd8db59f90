#!/usr/bin/env python3
"""Benchmark of the block-causal attention hot path on one MI355X.

One step runs every row of the hot path once:
  training   : block-causal attention forward + backward at B=1 H=16 T=42240
               D=128, 16 chunks of 2640 tokens (3 latent frames x 880 tokens),
               the largest training configuration, whose throughput is `value`;
               and the same at B=2 H=12 T=10560 D=64, 8 chunks of 1320 tokens;
  streaming  : commit one 2640-token chunk to the 8-slot KV ring, evict down to a
               6-chunk window, re-shift the retained keys' temporal RoPE band by
               the evicted chunk's 3 latent-frame positions, and cached attention
               of 4 queued in-flight chunks (2640 tokens each, B=1 H=16 D=128)
               over that window.
Inputs are seeded synthetic N(0,1) bf16 tensors resident in HBM before timing.

Prints one JSON line.  `value` is the D=128 training forward+backward
throughput in useful TFLOP/s (4 P D forward + 10 P D backward, P = visible
query-key pairs), timed with HIP events on the launch stream over the K timed
steps.  Outside the timed steps: the cache-bound decode shapes, a 200-step
rollout, the paper's own shapes, the e4m3 variant, what the vendor libraries
reach on this card (a copy, a read, a bf16 GEMM) and the CPU oracle baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PEAK_FP8_TFLOPS = 5000.0    # MI355X dense fp8 MFMA


def pairs_block_causal(B, H, T, L):
    """Visible (query, key) pairs of block-causal attention."""
    n = -(-T // L)
    tot = 0
    for c in range(n):
        rows = min(T, (c + 1) * L) - c * L
        tot += rows * min(T, (c + 1) * L)
    return B * H * tot


def pairs_cached(B, H, w, L, nq, qlen, causal=True):
    per = 0
    for j in range(nq):
        per += qlen * (w * L + ((j + 1) if causal else 1) * qlen)
    return B * H * per


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing leg")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target oracle sample duration")
    return ap.parse_args()


def source_digest(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def read_traffic(kernel: str, digest: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, if it was
    taken on the current kernel source; None otherwise."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha") != digest:
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _oracle_threads() -> int:
    try:
        from threadpoolctl import threadpool_info
        return int(max([i.get("num_threads", 1) for i in threadpool_info()] or [1]))
    except Exception:  # pragma: no cover
        return len(os.sched_getaffinity(0))


def cpu_baseline(target_s: float, d128_bits=None):
    """The fp64 oracle, as it stands, timed on bounded samples of the three
    headline workloads (about target_s seconds in all), each rate counted
    with the same useful-FLOP rule as the GPU (14 P D for forward+backward,
    4 P D for the cached call, P = visible pairs of the rows done):
      - B1 H16 T42240 D128 L2640 training: evenly spaced 512-row query blocks of
        head 0, each through the oracle's one-head forward and backward (the
        work the whole-sequence functions do per row block); extrapolated from
        those rows of one head;
      - B2 H12 T10560 D64 L1320 training: whole heads;
      - the cached call (4 queued 2640-token chunks over 6 committed chunks,
        H16 D128): whole heads.
    `value` is the D128 training sample's rate."""
    import numpy as np
    import oracle
    import synth
    threads = _oracle_threads()
    budget = {"d128": 0.45 * target_s, "d64": 0.3 * target_s, "cached": 0.25 * target_s}
    out = []

    # --- B1 H16 T42240 D128: 512-row blocks of head 0, evenly spaced
    s3 = synth.TRAIN_D128
    bits = d128_bits if d128_bits is not None else synth.training_inputs(s3)
    hq, hk, hv, hdo = (synth.bf16_bits_to_f64(bits[n][0, 0]) for n in ("q", "k", "v", "do"))
    sc = 1.0 / math.sqrt(s3.D)
    nblk = -(-s3.T // 512)
    order = []
    for stride in (16, 8, 4, 2, 1):  # coarse-to-fine sweep: every prefix is spread over the sequence
        order += [b for b in range(0, nblk, stride) if b not in order]
    pairs = blocks = 0
    t0 = time.perf_counter()
    for blk in order:
        rows = np.arange(blk * 512, min(s3.T, blk * 512 + 512))
        vis = oracle.block_causal_visible(rows, s3.T, s3.chunk_len)
        oracle.attention_fwd(hq[rows], hk, hv, vis, sc)
        oracle.attention_bwd(hq[rows], hk, hv, hdo[rows], vis, sc)
        pairs += int(vis.sum())
        blocks += 1
        if time.perf_counter() - t0 >= budget["d128"]:
            break
    dt = time.perf_counter() - t0
    out.append({"workload": s3.name, "value": round(14.0 * pairs * s3.D / dt / 1e12, 6), "unit": "TFLOP/s",
                "seconds": round(dt, 2),
                "sample": f"{blocks} of {nblk} evenly spaced 512-row query blocks of head 0 of 16, fwd+bwd, "
                          f"extrapolated from one head"})

    # --- B2 H12 T10560 D64: whole heads
    s2 = synth.TRAIN_D64
    b2 = synth.training_inputs(s2)
    t2 = {n: synth.bf16_bits_to_f64(b2[n]) for n in b2}
    heads = 0
    t0 = time.perf_counter()
    for b in range(s2.B):
        for h in range(s2.H):
            sl = (slice(b, b + 1), slice(h, h + 1))
            q, k, v, do = (t2[n][sl] for n in ("q", "k", "v", "do"))
            oracle.block_causal_attn_fwd(q, k, v, s2.chunk_len)
            oracle.block_causal_attn_bwd(q, k, v, do, s2.chunk_len)
            heads += 1
            if time.perf_counter() - t0 >= budget["d64"]:
                break
        if time.perf_counter() - t0 >= budget["d64"]:
            break
    dt = time.perf_counter() - t0
    flops = 14.0 * pairs_block_causal(1, heads, s2.T, s2.chunk_len) * s2.D
    out.append({"workload": s2.name, "value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s", "seconds": round(dt, 2),
                "sample": f"fwd+bwd of {heads} of {s2.B * s2.H} whole heads"})

    # --- cached call: whole heads of the streaming step
    st = synth.STREAM
    sb = synth.stream_step_inputs(st, 0, which=("q", "k_new", "v_new"))
    win = [synth.stream_step_inputs(st, i % 4, which=("k_commit", "v_commit")) for i in range(st.window)]
    heads = 0
    t0 = time.perf_counter()
    for h in range(st.H):
        sl = (slice(0, 1), slice(h, h + 1))
        q, kn, vn = (synth.bf16_bits_to_f64(sb[n][sl]) for n in ("q", "k_new", "v_new"))
        wk = [synth.bf16_bits_to_f64(w["k_commit"][sl]) for w in win]
        wv = [synth.bf16_bits_to_f64(w["v_commit"][sl]) for w in win]
        oracle.cached_chunk_attn(q, kn, vn, wk, wv, st.n_queued, st.q_len)
        heads += 1
        if time.perf_counter() - t0 >= budget["cached"]:
            break
    dt = time.perf_counter() - t0
    flops = 4.0 * pairs_cached(1, heads, st.window, st.chunk_len, st.n_queued, st.q_len) * st.D
    out.append({"workload": st.name + " cached call", "value": round(flops / dt / 1e12, 6), "unit": "TFLOP/s",
                "seconds": round(dt, 2), "sample": f"{heads} of {st.B * st.H} whole heads"})

    head = out[0]
    return {"value": head["value"], "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "sample": f"fp64 numpy oracle on {s3.name}: {head['sample']} ({head['seconds']} s), useful-FLOP "
                      f"count as the GPU; the other headline workloads in by_config",
            "by_config": out}


def decode_shapes(mw, torch, cache, st, dev, reps=20):
    """Cache-bound shapes: one queued chunk of 64 / 128 / 256 / 512 tokens over the full window
    (6 committed chunks of 2640 tokens, B1 H16 D128).  Each timed call is
    preceded by a 512 MB read (a sum) that evicts the 256 MB Infinity Cache, so
    the window's K/V come from HBM; a read leaves no dirty lines whose
    write-back would compete with the timed call.  Algorithmic bytes = window K
    and V + Q, K_new, V_new and O of the queued chunk."""
    out = []
    flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)
    g = torch.Generator(device=dev).manual_seed(1234)
    for ql in (64, 128, 256, 512):
        q, kn, vn = (torch.randn(st.B, st.H, ql, st.D, device=dev, generator=g).to(torch.bfloat16) for _ in range(3))
        o = torch.empty_like(q)
        ws = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(cache, 1, ql, st.window)), dtype=torch.uint8,
                         device=dev)
        run = lambda: mw.mw_chunk_attn_cached(q, kn, vn, 1, ql, cache, window=st.window, out=o, workspace=ws)
        for _ in range(3):
            run()
        tot = 0.0
        for _ in range(reps):
            flush.sum()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            run()
            e1.record()
            torch.cuda.synchronize()
            tot += e0.elapsed_time(e1)
        ms = tot / reps
        nbytes = 2 * st.window * st.B * st.H * st.chunk_len * st.D * 2 + 4 * st.B * st.H * ql * st.D * 2
        gbs = nbytes / (ms * 1e-3) / 1e9
        out.append({"q_len": ql, "us": round(ms * 1e3, 2), "gbs": round(gbs, 1),
                    "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "bytes": nbytes})
    return out


def library_ceilings(torch, dev, reps=20):
    """What the vendor libraries reach on this card, measured live beside the kernels (context for the
    rooflines, which stay on the published peaks): a 1 GiB device-to-device copy (bytes read plus
    written), a 1 GiB read (a sum), and a bf16 GEMM of 8192 x 8192 x 8192 through torch.matmul
    (hipBLASLt).  Each is the median of `reps` event-timed calls after 3 warm-up calls."""
    def med(fn):
        for _ in range(3):
            fn()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return sorted(ts)[len(ts) // 2]

    n = 1 << 28  # fp32 elements: 1 GiB
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    ms_copy = med(lambda: dst.copy_(src))
    ms_read = med(lambda: src.sum())
    del dst
    m = 8192
    g = torch.Generator(device=dev).manual_seed(4321)
    a = torch.randn(m, m, device=dev, generator=g).to(torch.bfloat16)
    b = torch.randn(m, m, device=dev, generator=g).to(torch.bfloat16)
    ms_gemm = med(lambda: torch.matmul(a, b))
    del src, a, b
    copy_gbs = 2 * 4 * n / (ms_copy * 1e-3) / 1e9
    read_gbs = 4 * n / (ms_read * 1e-3) / 1e9
    gemm_tf = 2.0 * m ** 3 / (ms_gemm * 1e-3) / 1e12
    return {"copy_1gib": {"gbs": round(copy_gbs, 1), "frac_hbm_peak": round(copy_gbs / PEAK_HBM_GBS, 4),
                          "us": round(ms_copy * 1e3, 1)},
            "read_1gib_sum": {"gbs": round(read_gbs, 1), "frac_hbm_peak": round(read_gbs / PEAK_HBM_GBS, 4),
                              "us": round(ms_read * 1e3, 1)},
            "gemm_bf16_8192": {"tflops": round(gemm_tf, 1), "frac_bf16_peak": round(gemm_tf / PEAK_BF16_TFLOPS, 4),
                               "us": round(ms_gemm * 1e3, 1)}}


def paper_shapes(mw, torch, dev, reps=5):
    """The paper's own 1B shapes (12 heads of width 128, 600-token chunks of 2
    latent frames): training forward+backward over a 32-chunk window (and the
    same with the 0.5B model's 16 heads of width 72), and
    cached attention of 8 in-flight chunks over 24/12/6 cached chunks plus a
    300-token sink with the guidance batch of 2, inputs as [B,T,H,D] views.
    Useful TFLOP/s, HIP events on the launch stream."""
    import synth
    out = {}
    tr = synth.PAPER_1B_TRAIN
    B, H, T, D, L = tr.B, tr.H, tr.T, tr.D, tr.chunk_len
    g = torch.Generator(device=dev).manual_seed(6)
    q, k, v, do = (torch.randn(B, H, T, D, device=dev, generator=g).to(torch.bfloat16) for _ in range(4))
    o = torch.empty_like(q)
    lse = torch.empty((B, H, T), dtype=torch.float32, device=dev)
    ws = torch.empty(mw.mw_block_causal_attn_bwd_workspace_size(B, H, T, D), dtype=torch.uint8, device=dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)

    def timed(fn):
        for _ in range(2):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    P = pairs_block_causal(B, H, T, L)
    tf = timed(lambda: mw.mw_block_causal_attn_fwd(q, k, v, L, out=o, lse=lse))
    tb = timed(lambda: mw.mw_block_causal_attn_bwd(q, k, v, o, do, lse, L, workspace=ws, dq=dq, dk=dk, dv=dv))
    out["train"] = {"workload": tr.name, "fwd_ms": round(tf, 4), "bwd_ms": round(tb, 4),
                    "fwd_bwd_tflops": round(14.0 * P * D / ((tf + tb) * 1e-3) / 1e12, 2)}
    # the 0.5B model's heads: 16 of width 72, same chunks and window
    H5, D5 = 16, 72
    q5, k5, v5, do5 = (torch.randn(B, H5, T, D5, device=dev, generator=g).to(torch.bfloat16) for _ in range(4))
    o5 = torch.empty_like(q5)
    lse5 = torch.empty((B, H5, T), dtype=torch.float32, device=dev)
    ws5 = torch.empty(mw.mw_block_causal_attn_bwd_workspace_size(B, H5, T, D5), dtype=torch.uint8, device=dev)
    g5 = [torch.empty_like(q5) for _ in range(3)]
    tf5 = timed(lambda: mw.mw_block_causal_attn_fwd(q5, k5, v5, L, out=o5, lse=lse5))
    tb5 = timed(lambda: mw.mw_block_causal_attn_bwd(q5, k5, v5, o5, do5, lse5, L, workspace=ws5, dq=g5[0], dk=g5[1],
                                                    dv=g5[2]))
    P5 = pairs_block_causal(B, H5, T, L)
    out["train_05b"] = {"workload": f"paper05b_train_B{B}H{H5}T{T}D{D5}L{L}", "fwd_ms": round(tf5, 4),
                        "bwd_ms": round(tb5, 4),
                        "fwd_bwd_tflops": round(14.0 * P5 * D5 / ((tf5 + tb5) * 1e-3) / 1e12, 2)}
    st = synth.PAPER_1B_STREAM
    B, H, D, L, nq = st.B, st.H, st.D, st.chunk_len, st.n_queued
    Tq = nq * st.q_len
    sk, sv = (torch.randn(B, H, st.sink_len, D, device=dev, generator=g).to(torch.bfloat16) for _ in range(2))
    qb, kb, vb = (torch.randn(B, Tq, H, D, device=dev, generator=g).to(torch.bfloat16) for _ in range(3))
    qv, kv, vv = (x.transpose(1, 2) for x in (qb, kb, vb))
    ob = torch.empty_like(qb)
    streams = []
    for window in (24, 12, 6):
        cache = mw.KVCache(window + 1, B, H, L, D, device=dev)
        kc = torch.randn(B, H, L, D, device=dev, generator=g).to(torch.bfloat16)
        for _ in range(window):
            mw.mw_kvcache_append(cache, kc, kc)
        cache.set_sink(sk, sv)
        wsb = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(cache, nq, st.q_len, window)),
                          dtype=torch.uint8, device=dev)
        tc = timed(lambda: mw.mw_chunk_attn_cached(qv, kv, vv, nq, st.q_len, cache, window=window,
                                                   out=ob.transpose(1, 2), workspace=wsb))
        hist = st.sink_len + window * L
        pairs = B * H * sum(st.q_len * (hist + (j + 1) * st.q_len) for j in range(nq))
        streams.append({"window": window, "ms": round(tc, 4), "tflops": round(4.0 * pairs * D / (tc * 1e-3) / 1e12, 2)})
    out["stream"] = {"workload": st.name.replace("_W24_S25", ""), "B_cfg": B, "by_window": streams}
    return out


def fp8_stream(mw, torch, dev, st, reps=10):
    """The e4m3 inference variant on the streaming shape (B1 H16 D128, 4 in-flight
    chunks of 2640 tokens over a 6-chunk window of an 8-slot ring): per step,
    quantize the queued chunks' Q, K, V (bf16 -> e4m3), commit one chunk
    (quantize-on-commit), evict to the window, re-shift the retained keys by the
    evicted chunk's 3 positions (recorded; the keys are rotated when the call
    loads the window), and run the e4m3 cached attention.
    Also the cache-bound decode shapes (one queued chunk of 64 / 128 / 256 tokens
    over the full window, Infinity Cache flushed before each call; algorithmic
    bytes = e4m3 window K and V + e4m3 Q, K_new, V_new + bf16 O), with nothing
    pending and with one re-shift pending (the window keys rotated as they are
    loaded, in the attention kernel's staging: one query tile per head), and
    the paper's
    1B streaming shape (CFG batch 2, 8 in-flight 600-token chunks, 300-token sink)
    over 24 / 12 / 6 cached chunks.  HIP events on the launch stream."""
    import synth
    B, H, D, L, nq, ql, W = st.B, st.H, st.D, st.chunk_len, st.n_queued, st.q_len, st.window
    sc = 5.0 / 448.0   # per-tensor scale for unit-variance activations
    g = torch.Generator(device=dev).manual_seed(8)
    cache = mw.KVCache(st.slots, B, H, L, D, device=dev, fp8=True, k_scale=sc, v_scale=sc)
    kc = torch.randn(B, H, L, D, device=dev, generator=g).to(torch.bfloat16)
    vc = torch.randn(B, H, L, D, device=dev, generator=g).to(torch.bfloat16)
    for _ in range(W):
        mw.mw_kvcache_append(cache, kc, vc)
    Tq = nq * ql
    qb, kb, vb = (torch.randn(B, H, Tq, D, device=dev, generator=g).to(torch.bfloat16) for _ in range(3))
    q8, k8, v8 = (torch.empty((B, H, Tq, D), dtype=torch.uint8, device=dev) for _ in range(3))
    o = torch.empty_like(qb)
    ws = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(cache, nq, ql, W)), dtype=torch.uint8, device=dev)

    def ev():
        e = torch.cuda.Event(enable_timing=True)
        e.record()
        return e

    ph = {"quantize_qkv": 0.0, "append": 0.0, "cached": 0.0}

    def step(rec):
        e0 = ev()
        for x, y in ((qb, q8), (kb, k8), (vb, v8)):
            mw.mw_quantize_fp8(x, sc, out=y)
        e1 = ev()
        mw.mw_kvcache_append(cache, kc, vc)
        e2 = ev()
        n_ev = cache.live - W
        mw.mw_kvcache_evict(cache, n_ev)
        mw.mw_kvcache_rope_shift(cache, 3 * n_ev, 0, 44)
        e3 = ev()
        mw.mw_chunk_attn_cached_fp8(q8, k8, v8, nq, ql, cache, sc, window=W, out=o, workspace=ws)
        e4 = ev()
        if rec is not None:
            rec.append((e0, e1, e2, e3, e4))

    for _ in range(3):
        step(None)
    torch.cuda.synchronize()
    recs = []
    for _ in range(reps):
        step(recs)
    torch.cuda.synchronize()
    for e in recs:
        ph["quantize_qkv"] += e[0].elapsed_time(e[1]) / reps
        ph["append"] += e[1].elapsed_time(e[2]) / reps
        ph["cached"] += e[3].elapsed_time(e[4]) / reps
    step_ms = sum(e[0].elapsed_time(e[4]) for e in recs) / reps
    F = 4.0 * pairs_cached(B, H, W, L, nq, ql, causal=True) * D
    n_el = B * H * Tq * D
    out = {"workload": st.name + "_e4m3", "dtype": "e4m3 (fp32 accumulate)", "scale": sc,
           "rope": "re-shift of 3 positions per step, rotated on load (inside the cached call)",
           "step_ms": round(step_ms, 4),
           "phases_ms": {k: round(v, 4) for k, v in ph.items()},
           "cached_tflops": round(F / (ph["cached"] * 1e-3) / 1e12, 2),
           "cached_frac_fp8_peak": round(F / (ph["cached"] * 1e-3) / 1e12 / PEAK_FP8_TFLOPS, 4),
           "step_tflops": round(F / (step_ms * 1e-3) / 1e12, 2),
           "quantize_qkv_gbs": round(3 * n_el * 3 / (ph["quantize_qkv"] * 1e-3) / 1e9, 1),
           "append_gbs": round(2 * B * H * L * D * 3 / (ph["append"] * 1e-3) / 1e9, 1)}
    # decode shapes: on a cache of the same window with no shift pending (pure
    # streaming of the window), and after one re-shift (the state of a rollout
    # between evictions: the window keys are rotated as the call loads them)
    flush = torch.ones(128 << 20, dtype=torch.float32, device=dev)
    for key, shift in (("decode", 0), ("decode_shift_pending", 3)):
        cache = mw.KVCache(st.slots, B, H, L, D, device=dev, fp8=True, k_scale=sc, v_scale=sc)
        for _ in range(W):
            mw.mw_kvcache_append(cache, kc, vc)
        if shift:
            mw.mw_kvcache_rope_shift(cache, shift, 0, 44)
        dec = []
        for dq in (64, 128, 256):
            q1, k1, v1 = (torch.randint(0, 120, (B, H, dq, D), dtype=torch.uint8, device=dev, generator=g)
                          for _ in range(3))
            o1 = torch.empty((B, H, dq, D), dtype=torch.bfloat16, device=dev)
            ws1 = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(cache, 1, dq, W)), dtype=torch.uint8,
                              device=dev)
            run = lambda: mw.mw_chunk_attn_cached_fp8(q1, k1, v1, 1, dq, cache, sc, window=W, out=o1, workspace=ws1)
            for _ in range(3):
                run()
            tot = 0.0
            for _ in range(reps):
                flush.sum()
                e0 = ev()
                run()
                e1 = ev()
                torch.cuda.synchronize()
                tot += e0.elapsed_time(e1)
            ms = tot / reps
            nbytes = 2 * W * B * H * L * D + 3 * B * H * dq * D + B * H * dq * D * 2
            gbs = nbytes / (ms * 1e-3) / 1e9
            dec.append({"q_len": dq, "us": round(ms * 1e3, 2), "gbs": round(gbs, 1),
                        "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "bytes": nbytes})
        out[key] = dec
    # the paper's 1B streaming shape
    ps = synth.PAPER_1B_STREAM
    B, H, D, L, nq = ps.B, ps.H, ps.D, ps.chunk_len, ps.n_queued
    Tq = nq * ps.q_len
    s8 = [torch.randint(0, 120, (B, H, ps.sink_len, D), dtype=torch.uint8, device=dev, generator=g) for _ in range(2)]
    x8 = [torch.randint(0, 120, (B, H, Tq, D), dtype=torch.uint8, device=dev, generator=g) for _ in range(3)]
    ob = torch.empty((B, Tq, H, D), dtype=torch.bfloat16, device=dev)
    kc = torch.randn(B, H, L, D, device=dev, generator=g).to(torch.bfloat16)
    by = []
    for window in (24, 12, 6):
        c8 = mw.KVCache(window + 1, B, H, L, D, device=dev, fp8=True, k_scale=sc, v_scale=sc)
        for _ in range(window):
            mw.mw_kvcache_append(c8, kc, kc)
        c8.set_sink(*s8)
        wsb = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(c8, nq, ps.q_len, window)),
                          dtype=torch.uint8, device=dev)
        fn = lambda: mw.mw_chunk_attn_cached_fp8(*x8, nq, ps.q_len, c8, sc, window=window, out=ob.transpose(1, 2),
                                                 workspace=wsb)
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0 = ev()
        for _ in range(reps):
            fn()
        e1 = ev()
        torch.cuda.synchronize()
        tc = e0.elapsed_time(e1) / reps
        hist = ps.sink_len + window * L
        pairs = B * H * sum(ps.q_len * (hist + (j + 1) * ps.q_len) for j in range(nq))
        by.append({"window": window, "ms": round(tc, 4), "tflops": round(4.0 * pairs * D / (tc * 1e-3) / 1e12, 2)})
    out["paper_1b_stream"] = {"workload": ps.name.replace("_W24_S25", "") + "_e4m3", "B_cfg": B, "by_window": by}
    return out


def rollout(mw, torch, dev, st, steps=200):
    """The long-horizon rollout: 200 chunk steps from an empty ring, each one
    commit (append), eviction down to the 6-chunk window, and cached attention
    of the 4 queued chunks over the live window (1, 2, ... 6 committed chunks,
    then 6 with the ring wrapping every 8 commits).  Timed as a whole with HIP
    events on the launch stream; useful TFLOP/s counts each step's visible
    pairs with its actual window."""
    g = torch.Generator(device=dev).manual_seed(5)
    B, H, D, L, nq, ql, W = st.B, st.H, st.D, st.chunk_len, st.n_queued, st.q_len, st.window
    cache = mw.KVCache(st.slots, B, H, L, D, device=dev)
    srcs = [tuple(torch.randn(B, H, L, D, device=dev, generator=g).to(torch.bfloat16) for _ in range(2))
            for _ in range(4)]
    q, kn, vn = (torch.randn(B, H, nq * ql, D, device=dev, generator=g).to(torch.bfloat16) for _ in range(3))
    o = torch.empty_like(q)
    ws = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(cache, nq, ql, W)), dtype=torch.uint8,
                     device=dev)
    windows = []

    def run(n, record):
        for t in range(n):
            mw.mw_kvcache_append(cache, *srcs[t % 4])
            mw.mw_kvcache_evict(cache, max(0, cache.live - W))
            mw.mw_chunk_attn_cached(q, kn, vn, nq, ql, cache, window=cache.live, out=o, workspace=ws)
            if record:
                windows.append(cache.live)

    run(8, False)  # warm-up on a scratch ring (plans memoised, code loaded)
    cache = mw.KVCache(st.slots, B, H, L, D, device=dev)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    run(steps, True)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    F = sum(4.0 * pairs_cached(B, H, w, L, nq, ql) * D for w in windows)
    return {"workload": synth_name(st, steps), "steps": steps, "total_ms": round(ms, 3),
            "ms_per_step": round(ms / steps, 4), "tflops": round(F / (ms * 1e-3) / 1e12, 2),
            "append_bytes_per_step": 4 * B * H * L * D * 2}


def synth_name(st, steps):
    return f"rollout_B{st.B}H{st.H}D{st.D}L{st.chunk_len}_nq{st.n_queued}_W{st.window}_S{st.slots}_{steps}steps"


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on exactly one GPU; --gpus must be 1 (the hot path is "
                                   "measured on one GPU's share; sharding is a design note only)"}))
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2608_01127_amd as mw
    import synth

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    mw.load()

    def up(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(dev)

    # ------------------------------------------------------------------ inputs (resident in HBM)
    class Train:
        """One training workload's tensors and useful FLOPs."""

        def __init__(self, shape, bits):
            self.s = shape
            self.q, self.k, self.v, self.do = (up(bits[n]) for n in ("q", "k", "v", "do"))
            B, H, T, D = shape.B, shape.H, shape.T, shape.D
            self.o = torch.empty_like(self.q)
            self.lse = torch.empty((B, H, T), dtype=torch.float32, device=dev)
            self.dq, self.dk, self.dv = (torch.empty_like(self.q) for _ in range(3))
            self.ws = torch.empty(mw.mw_block_causal_attn_bwd_workspace_size(B, H, T, D), dtype=torch.uint8,
                                  device=dev)
            P = pairs_block_causal(B, H, T, shape.chunk_len)
            self.F_fwd, self.F_bwd = 4.0 * P * D, 10.0 * P * D

        def fwd(self):
            mw.mw_block_causal_attn_fwd(self.q, self.k, self.v, self.s.chunk_len, out=self.o, lse=self.lse)

        def bwd(self):
            mw.mw_block_causal_attn_bwd(self.q, self.k, self.v, self.o, self.do, self.lse, self.s.chunk_len,
                                        workspace=self.ws, dq=self.dq, dk=self.dk, dv=self.dv)

    bits128 = synth.training_inputs(synth.TRAIN_D128)
    t128 = Train(synth.TRAIN_D128, bits128)   # the largest training configuration: the headline
    t64 = Train(synth.TRAIN_D64, synth.training_inputs(synth.TRAIN_D64))

    st = synth.STREAM
    cache = mw.KVCache(st.slots, st.B, st.H, st.chunk_len, st.D, device=dev)
    n_src = 4  # distinct commit sources, rotated
    commits = []
    for i in range(n_src):
        cb = synth.stream_step_inputs(st, i, which=("k_commit", "v_commit"))
        commits.append((up(cb["k_commit"]), up(cb["v_commit"])))
    sb = synth.stream_step_inputs(st, 0, which=("q", "k_new", "v_new"))
    sq, skn, svn = (up(sb[n]) for n in ("q", "k_new", "v_new"))
    so = torch.empty_like(sq)
    ws_c = torch.empty(max(16, mw.mw_chunk_attn_cached_workspace_size(cache, st.n_queued, st.q_len, st.window)),
                       dtype=torch.uint8, device=dev)
    for i in range(st.window):
        mw.mw_kvcache_append(cache, *commits[i % n_src])
    torch.cuda.synchronize()

    P_st = pairs_cached(st.B, st.H, st.window, st.chunk_len, st.n_queued, st.q_len, causal=True)
    F_st = 4.0 * P_st * st.D
    chunk_bytes = st.B * st.H * st.chunk_len * st.D * 2
    bytes_append = 4 * chunk_bytes                       # read K,V chunk + write K,V slot
    bytes_cached = (4 * st.B * st.H * st.n_queued * st.q_len * st.D * 2   # Q, K_new, V_new, O
                    + 2 * st.window * chunk_bytes)                         # window K, V

    ev = lambda: torch.cuda.Event(enable_timing=True)
    step_i = [0]

    rope_off, rope_cnt = 0, st.D - 4 * (st.D // 6)  # temporal rope band (reading: first D - 4*floor(D/6) dims)
    frames_per_chunk = 3
    bytes_rope = 2 * st.window * st.B * st.H * st.chunk_len * rope_cnt * 2  # band read + written

    PH = ["fwd_d128", "bwd_d128", "fwd_d64", "bwd_d64", "append", "rope_shift", "cached"]

    def step(rec=None):
        e = [ev() for _ in range(len(PH) + 1)] if rec is not None else None
        mark = (lambda i: e[i].record()) if e else (lambda i: None)
        mark(0)
        t128.fwd()
        mark(1)
        t128.bwd()
        mark(2)
        t64.fwd()
        mark(3)
        t64.bwd()
        mark(4)
        mw.mw_kvcache_append(cache, *commits[step_i[0] % n_src])
        step_i[0] += 1
        mark(5)
        n_ev = cache.live - st.window
        mw.mw_kvcache_evict(cache, n_ev)
        mw.mw_kvcache_rope_shift(cache, n_ev * frames_per_chunk, rope_off, rope_cnt)
        mark(6)
        mw.mw_chunk_attn_cached(sq, skn, svn, st.n_queued, st.q_len, cache, window=st.window,
                                flags=mw.MW_QUEUED_CAUSAL, out=so, workspace=ws_c)
        mark(7)
        if rec is not None:
            rec.append(e)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    recs = []
    t_start, t_end = ev(), ev()
    torch.cuda.synchronize()
    t_start.record()
    for _ in range(args.steps):
        step(recs)
    t_end.record()
    torch.cuda.synchronize()
    K = args.steps
    total_ms = t_start.elapsed_time(t_end)
    ph = {n: sum(e[i].elapsed_time(e[i + 1]) for e in recs) / K for i, n in enumerate(PH)}
    per_step = {n: sorted(e[i].elapsed_time(e[i + 1]) for e in recs) for i, n in enumerate(PH)}
    ph_median = {n: v[len(v) // 2] for n, v in per_step.items()}
    ph_min = {n: v[0] for n, v in per_step.items()}
    ms_step = total_ms / K
    tfl = lambda F, ms: F / (ms * 1e-3) / 1e12
    gbs = lambda nb, ms: nb / (ms * 1e-3) / 1e9
    value = tfl(t128.F_fwd + t128.F_bwd, ph["fwd_d128"] + ph["bwd_d128"])
    value64 = tfl(t64.F_fwd + t64.F_bwd, ph["fwd_d64"] + ph["bwd_d64"])
    cached_tflops = tfl(F_st, ph["cached"])
    n_splits, n_whole = mw.mw_chunk_attn_cached_plan(cache, st.n_queued, st.q_len, st.window, 0, ws_c.numel())

    # Dominant launch of the step: the D128 training backward call
    # (mw_block_causal_attn_bwd: the row terms, then the dK/dV and dQ work in
    # one grid).  Its algorithmic FLOPs are the backward's useful 10 P D; the
    # events bracket both kernels, so the duration is the call's.
    bwd_digest = source_digest(["paper_2608_01127_amd/csrc/attn_bwd.hip", "paper_2608_01127_amd/csrc/mw_device.h",
                                "paper_2608_01127_amd/csrc/mw_kernels.h", "paper_2608_01127_amd/build.py"])
    roofline = {"kernel": "mw_block_causal_attn_bwd at B1 H16 T42240 D128 L2640 = bwd_rowterms_kernel<128> + "
                          "bwd_grad_kernel<128, 4, 32, 4, 1, 64, true>",
                "bound": "mfma", "achieved": round(tfl(t128.F_bwd, ph["bwd_d128"]), 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(tfl(t128.F_bwd, ph["bwd_d128"]) / PEAK_BF16_TFLOPS, 4),
                "traffic": read_traffic("train_bwd_d128", bwd_digest),
                "algorithmic_flops_per_launch": t128.F_bwd, "avg_launch_ms": round(ph["bwd_d128"], 4)}

    def mf(name, F, ms):
        a = tfl(F, ms)
        return {"phase": name, "bound": "mfma", "achieved": round(a, 2), "unit": "TFLOP/s", "peak": PEAK_BF16_TFLOPS,
                "frac": round(a / PEAK_BF16_TFLOPS, 4), "ms": round(ms, 4)}

    def hb(name, nb, ms):
        a = gbs(nb, ms)
        return {"phase": name, "bound": "hbm", "achieved": round(a, 1), "unit": "GB/s", "peak": PEAK_HBM_GBS,
                "frac": round(a / PEAK_HBM_GBS, 4), "ms": round(ms, 4)}

    fwd_digest = source_digest(["paper_2608_01127_amd/csrc/attn_fwd.hip", "paper_2608_01127_amd/csrc/mw_device.h",
                                "paper_2608_01127_amd/csrc/mw_kernels.h", "paper_2608_01127_amd/build.py"])
    cached_rl = mf("cached chunk attention call", F_st, ph["cached"])
    cached_rl["traffic"] = read_traffic("attn_fwd_cached", fwd_digest)
    cached_rl["n_splits"], cached_rl["n_whole"] = n_splits, n_whole
    rooflines = [mf("train fwd D128", t128.F_fwd, ph["fwd_d128"]), mf("train bwd D128", t128.F_bwd, ph["bwd_d128"]),
                 mf("train fwd D64", t64.F_fwd, ph["fwd_d64"]), mf("train bwd D64", t64.F_bwd, ph["bwd_d64"]),
                 cached_rl, hb("append (commit)", bytes_append, ph["append"]),
                 hb("rope re-shift", bytes_rope, ph["rope_shift"])]

    s3, s2 = synth.TRAIN_D128, synth.TRAIN_D64
    res = {
        "metric": "block-causal attn fwd+bwd TFLOP/s (% bf16 MFMA peak); cached-chunk attn GB/s",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{s3.name} fwd+bwd (value) + {s2.name} fwd+bwd + {st.name} streaming step",
                   "train": {"B": s3.B, "H": s3.H, "T": s3.T, "D": s3.D, "chunk_len": s3.chunk_len},
                   "train_d64": {"B": s2.B, "H": s2.H, "T": s2.T, "D": s2.D, "chunk_len": s2.chunk_len},
                   "stream": {"B": st.B, "H": st.H, "D": st.D, "chunk_len": st.chunk_len, "n_queued": st.n_queued,
                              "q_len": st.q_len, "window": st.window, "slots": st.slots,
                              "visibility": "queued-causal"}},
        "frac_bf16_peak": round(value / PEAK_BF16_TFLOPS, 4),
        "phases_ms": {n: round(t, 4) for n, t in ph.items()},
        "phases_ms_median": {n: round(t, 4) for n, t in ph_median.items()},
        "phases_ms_min": {n: round(t, 4) for n, t in ph_min.items()},
        "train_d128": {"fwd_tflops": round(tfl(t128.F_fwd, ph["fwd_d128"]), 2),
                       "bwd_tflops": round(tfl(t128.F_bwd, ph["bwd_d128"]), 2), "fwd_bwd_tflops": round(value, 2)},
        "train_d64": {"fwd_tflops": round(tfl(t64.F_fwd, ph["fwd_d64"]), 2),
                      "bwd_tflops": round(tfl(t64.F_bwd, ph["bwd_d64"]), 2), "fwd_bwd_tflops": round(value64, 2),
                      "frac_bf16_peak": round(value64 / PEAK_BF16_TFLOPS, 4)},
        "cached_attn": {"tflops": round(cached_tflops, 2), "gbs": round(gbs(bytes_cached, ph["cached"]), 1),
                        "frac_bf16_peak": round(cached_tflops / PEAK_BF16_TFLOPS, 4)},
        "append": {"gbs": round(gbs(bytes_append, ph["append"]), 1),
                   "frac_hbm_peak": round(gbs(bytes_append, ph["append"]) / PEAK_HBM_GBS, 4)},
        "rope_shift": {"positions": frames_per_chunk, "band": [rope_off, rope_off + rope_cnt],
                       "gbs": round(gbs(bytes_rope, ph["rope_shift"]), 1),
                       "frac_hbm_peak": round(gbs(bytes_rope, ph["rope_shift"]) / PEAK_HBM_GBS, 4)},
        "roofline": roofline,
        "rooflines": rooflines,
    }
    res["decode"] = decode_shapes(mw, torch, cache, st, dev)
    res["rollout"] = rollout(mw, torch, dev, st)
    res["paper_1b"] = paper_shapes(mw, torch, dev)
    res["fp8_stream"] = fp8_stream(mw, torch, dev, st)
    res["library_ceilings"] = library_ceilings(torch, dev)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(args.cpu_seconds, bits128)
    else:
        res["cpu_baseline"] = None
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()

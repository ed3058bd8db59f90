"""Host-side checks of the C ABI: the library loads, exports every declared symbol, validates
arguments before touching the device, and keeps ring bookkeeping that agrees with the ring model.

Only calls that return before any HIP call are made (no GPU is needed).  Pointers passed here are
fake host addresses that are never dereferenced.
"""
import ctypes
import os
import re

import pytest

import oracle
import paper_2608_01127_amd as mw
from paper_2608_01127_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
A = 0x10000   # aligned fake pointer
U = 0x10008   # misaligned fake pointer


def declared_functions():
    text = open(os.path.join(ROOT, "include", "mw.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mw_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = mw.load()
    names = declared_functions()
    assert len(names) >= 10
    for n in names:
        assert hasattr(lib, n), n
        assert n in _lib.SIGNATURES, f"binding lacks {n}"
    assert lib.mw_version() == 100


def test_struct_layout_matches_header():
    assert ctypes.sizeof(_lib.mw_kvcache) == 112 + 8 * _lib.MW_MAX_SLOTS
    assert _lib.mw_kvcache.head.offset == 40 and _lib.mw_kvcache.tail.offset == 48
    assert _lib.mw_kvcache.k_sink.offset == 56 and _lib.mw_kvcache.sink_len.offset == 72
    assert _lib.mw_kvcache.elem_bytes.offset == 76 and _lib.mw_kvcache.v_scale.offset == 84
    assert _lib.mw_kvcache.rope_total.offset == 88 and _lib.mw_kvcache.rope_set.offset == 108
    assert _lib.mw_kvcache.rope_at_commit.offset == 112
    text = open(os.path.join(ROOT, "include", "mw.h")).read()
    assert re.search(r"#define MW_MAX_SLOTS %d\b" % _lib.MW_MAX_SLOTS, text)
    assert ctypes.sizeof(_lib.mw_rope) == 12


def err():
    return mw.load().mw_last_error().decode()


def test_fwd_validation():
    lib = mw.load()
    f = lib.mw_block_causal_attn_fwd
    assert f(None, A, A, A, A, 1, 1, 64, 64, 16, 0.125, None) == mw.MW_EINVAL and "q is NULL" in err()
    assert f(A, A, U, A, A, 1, 1, 64, 64, 16, 0.125, None) == mw.MW_EALIGN and "v" in err()
    assert f(A, A, A, A, A, 1, 1, 64, 96, 16, 0.125, None) == mw.MW_EUNSUPPORTED
    assert f(A, A, A, A, A, 1, 1, 64, 64, 0, 0.125, None) == mw.MW_EINVAL
    assert f(A, A, A, A, A, 0, 1, 64, 64, 4, 0.125, None) == mw.MW_EINVAL
    assert f(A, A, A, A, A, 1, 1, 0, 64, 4, 0.125, None) == mw.MW_EINVAL
    assert f(A, A, A, A, A, 1, 1, 64, 64, 4, 0.0, None) == mw.MW_EINVAL
    assert f(A, A, A, A, A, 1, 1, 64, 64, 4, float("nan"), None) == mw.MW_EINVAL


def test_bwd_validation_and_workspace():
    lib = mw.load()
    ws = lib.mw_block_causal_attn_bwd_workspace_size(2, 3, 100, 64)
    assert ws >= 2 * 3 * 100 * 4 and ws % 256 == 0
    assert lib.mw_block_causal_attn_bwd_workspace_size(0, 3, 100, 64) == 0
    b = lib.mw_block_causal_attn_bwd
    args = [A] * 10
    assert b(*args, ws - 1, 2, 3, 100, 64, 10, 0.125, None) == mw.MW_EINVAL and "workspace" in err()
    bad = list(args)
    bad[4] = None
    assert b(*bad, ws, 2, 3, 100, 64, 10, 0.125, None) == mw.MW_EINVAL
    bad[4] = U
    assert b(*bad, ws, 2, 3, 100, 64, 10, 0.125, None) == mw.MW_EALIGN
    assert b(*args, ws, 2, 3, 100, 32, 10, 0.125, None) == mw.MW_EUNSUPPORTED


def strides(*triples):
    arr = (_lib.mw_strides * len(triples))()
    for i, t in enumerate(triples):
        arr[i] = _lib.mw_strides(*t)
    return arr


def test_strided_validation():
    """Views: strides >= 0, multiples of 8 elements, T stride >= D; outputs must not overlap
    themselves.  Every call here fails validation, so nothing is launched."""
    lib = mw.load()
    f = lib.mw_block_causal_attn_fwd_strided
    B, H, T, D = 2, 3, 40, 64
    cont = (H * T * D, T * D, D)
    bthd = (T * H * D, D, H * D)             # [B,T,H,D] seen as [B,H,T,D]
    fused = (3 * T * H * D, D, 3 * H * D)    # q/k/v inside [B,T,3,H,D]
    # valid input views get past the stride checks and stop at a bad output view
    for good in (cont, bthd, fused):
        st = strides(good, good, good, (H * T * D, D, D))
        assert f(A, A, A, A, A, st, B, H, T, D, 8, 0.125, None) == mw.MW_EINVAL and "o overlaps" in err()
    bad_cases = [
        (strides((-8, T * D, D), cont, cont, cont), mw.MW_EINVAL, "strides of q"),
        (strides(cont, (H * T * D, T * D, 60), cont, cont), mw.MW_EINVAL, "strides of k"),
        (strides(cont, cont, (H * T * D, T * D + 4, D + 4), cont), mw.MW_EALIGN, "multiples of 8"),
        (strides(cont, cont, cont, (H * T * D, D, D)), mw.MW_EINVAL, "overlaps"),
        (strides(cont, cont, cont, (0, T * D, D)), mw.MW_EINVAL, "overlaps"),
    ]
    for st, code, msg in bad_cases:
        assert f(A, A, A, A, A, st, B, H, T, D, 8, 0.125, None) == code, msg
        assert msg in err()
    # inputs may broadcast (stride 0) and overlap each other; outputs may not overlap themselves
    bwd = lib.mw_block_causal_attn_bwd_strided
    ws = lib.mw_block_causal_attn_bwd_workspace_size(B, H, T, D)
    st8 = strides(cont, cont, cont, cont, cont, cont, (H * T * D, D, D), cont)
    assert bwd(*([A] * 10), ws, st8, B, H, T, D, 8, 0.125, None) == mw.MW_EINVAL and "dk overlaps" in err()
    c = new_cache(S=4, B=1, H=2, L=16, D=64)
    ap = lib.mw_kvcache_append_strided
    assert ap(ctypes.byref(c), A, A, strides((2 * 16 * 64, 16 * 64, 63), (2 * 16 * 64, 16 * 64, 64)), None) \
        == mw.MW_EINVAL and c.head == 0
    ca = lib.mw_chunk_attn_cached_strided
    st4 = strides(cont, cont, cont, (0, 0, 64))
    assert ca(A, A, A, 1, 16, ctypes.byref(c), 0, 0, A, None, 0.125, None, 0, st4, None) == mw.MW_EINVAL


def new_cache(S=8, B=1, H=2, L=16, D=64):
    c = _lib.mw_kvcache()
    assert mw.load().mw_kvcache_init(ctypes.byref(c), A, A, S, B, H, L, D) == mw.MW_OK
    return c


def test_kvcache_init_validation():
    lib = mw.load()
    c = _lib.mw_kvcache()
    assert lib.mw_kvcache_init(None, A, A, 8, 1, 1, 16, 64) == mw.MW_EINVAL
    assert lib.mw_kvcache_init(ctypes.byref(c), A, U, 8, 1, 1, 16, 64) == mw.MW_EALIGN
    assert lib.mw_kvcache_init(ctypes.byref(c), A, A, 0, 1, 1, 16, 64) == mw.MW_EINVAL
    assert lib.mw_kvcache_init(ctypes.byref(c), A, A, 8, 1, 1, 16, 80) == mw.MW_EUNSUPPORTED
    c = new_cache()
    assert (c.head, c.tail, c.S, c.L, c.D) == (0, 0, 8, 16, 64)


def test_ring_bookkeeping_matches_model_300_steps():
    """Commits are simulated by advancing `head` (the device copy is not run without a GPU);
    eviction, live counts and slot lookup go through the C ABI and must match the model."""
    lib = mw.load()
    S, W = 8, 6
    c = new_cache(S=S)
    ring = oracle.RingModel(S)
    for t in range(300):
        ring.append()
        c.head += 1
        if ring.live > W:
            n = ring.live - W
            ring.evict(n)
            assert lib.mw_kvcache_evict(ctypes.byref(c), n) == mw.MW_OK
        assert lib.mw_kvcache_live(ctypes.byref(c)) == ring.live
        for chunk in range(max(0, t - 12), t + 3):
            assert lib.mw_kvcache_slot_of(ctypes.byref(c), chunk) == ring.slot_of(chunk)
    assert (c.head, c.tail) == (ring.head, ring.tail)


def test_ring_full_empty_and_window_errors():
    lib = mw.load()
    c = new_cache(S=3)
    c.head = 3  # three live chunks: the ring is full
    assert lib.mw_kvcache_append(ctypes.byref(c), A, A, None) == mw.MW_EFULL and "evict" in err()
    assert c.head == 3
    assert lib.mw_kvcache_evict(ctypes.byref(c), 4) == mw.MW_EEMPTY
    assert lib.mw_kvcache_evict(ctypes.byref(c), -1) == mw.MW_EINVAL
    assert c.tail == 0
    cached = lambda *a: lib.mw_chunk_attn_cached(*a[:11], None, 0, None)
    assert cached(A, A, A, 2, 16, ctypes.byref(c), 4, 0, A, None, 0.125) == mw.MW_EINVAL and "window" in err()
    assert cached(A, A, A, 2, 16, ctypes.byref(c), -2, 0, A, None, 0.125) == mw.MW_EINVAL
    assert cached(A, A, A, 2, 16, ctypes.byref(c), 1, 7, A, None, 0.125) == mw.MW_EINVAL
    assert cached(A, A, A, 0, 16, ctypes.byref(c), 1, 0, A, None, 0.125) == mw.MW_EINVAL
    assert cached(A, A, A, 2, 16, ctypes.byref(c), 1, 0, A, U, 0.125) == mw.MW_EALIGN
    assert cached(A, None, A, 2, 16, ctypes.byref(c), 1, 0, A, None, 0.125) == mw.MW_EINVAL
    assert cached(A, A, A, 65, 16, ctypes.byref(c), 1, 0, A, None, 0.125) == mw.MW_EUNSUPPORTED
    assert lib.mw_chunk_attn_cached(A, A, A, 2, 16, ctypes.byref(c), 1, 0, A, None, 0.125, U, 1 << 20,
                                    None) == mw.MW_EALIGN
    # a corrupt descriptor is rejected
    c.tail = 5
    assert lib.mw_kvcache_evict(ctypes.byref(c), 0) == mw.MW_EINVAL
    assert lib.mw_kvcache_slot_of(None, 0) == -1


def test_cached_workspace_size_policy():
    """The split heuristic asks for workspace only when there are few query tiles."""
    lib = mw.load()
    c = new_cache(S=8, B=1, H=16, L=2640, D=128)
    c.head = 6
    assert lib.mw_chunk_attn_cached_workspace_size(None, 1, 64, -1) == 0
    big = lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), 4, 2640, 6)   # 42 tiles x 16 heads
    small = lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), 1, 128, 6)  # one tile per head
    # per split and split query row: fp32 O (D floats) plus (m, l)
    assert big % (16 * 130 * 4) == 0 and 0 < big < 8 * 16 * 4 * 2640 * 130 * 4
    assert small % (16 * 128 * 130 * 4) == 0 and small // (16 * 128 * 130 * 4) >= 8
    assert lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), 0, 128, 6) == 0


# Split plans over a 6 x 2640-token window (B1 H16 D128), queued-causal, as
# (key ranges, whole tiles per head).  Measured on MI355X: the uniform counts
# are the fastest of 1-8 splits (1024-2640 queued rows) and of 4-32 (one chunk
# of 64-512 rows); four 2640-token chunks (42 query tiles per head) run their
# 32 heaviest tiles unsplit and the first chunk's 10 tiles over 3 key ranges.
@pytest.mark.parametrize("e4m3, n_queued, q_len, plan", [
    (False, 4, 2640, (3, 32)), (False, 1, 2640, (4, 0)), (False, 1, 1024, (4, 0)), (False, 1, 64, (16, 0)),
    (False, 1, 128, (16, 0)), (False, 1, 256, (8, 0)), (False, 1, 512, (4, 0)), (True, 1, 64, (16, 0)),
    (True, 1, 128, (16, 0))])
def test_cached_split_plan(e4m3, n_queued, q_len, plan):
    lib = mw.load()
    if e4m3:
        c = _lib.mw_kvcache()
        assert lib.mw_kvcache_init_fp8(ctypes.byref(c), A, A, 8, 1, 16, 2640, 128, 0.02, 0.02) == mw.MW_OK
    else:
        c = new_cache(S=8, B=1, H=16, L=2640, D=128)
    c.head = 6
    ws = lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), n_queued, q_len, 6)
    ns, nw = ctypes.c_int(-1), ctypes.c_int(-1)
    assert lib.mw_chunk_attn_cached_plan(ctypes.byref(c), n_queued, q_len, 6, mw.MW_QUEUED_CAUSAL, ws,
                                         ctypes.byref(ns), ctypes.byref(nw)) == mw.MW_OK
    assert (ns.value, nw.value) == plan
    # the plan fits the workspace the library asks for; without one nothing is split
    bm = 64 if (q_len <= 64) else (128 if q_len <= (128 if e4m3 else 512) and n_queued * q_len <= 512 else 256)
    nqt = -(-n_queued * q_len // bm)
    rows = min(n_queued * q_len, (nqt - nw.value) * bm) if ns.value > 1 else 0
    assert ns.value * 16 * rows * 130 * 4 <= ws
    assert lib.mw_chunk_attn_cached_plan(ctypes.byref(c), n_queued, q_len, 6, mw.MW_QUEUED_CAUSAL, 0,
                                         ctypes.byref(ns), ctypes.byref(nw)) == mw.MW_OK
    assert (ns.value, nw.value) == (1, 0)


def test_small_hybrid_split_plans():
    """The small shapes the GPU parity tests use for plans with whole and split query tiles."""
    lib = mw.load()
    ns, nw = ctypes.c_int(), ctypes.c_int()
    for (H, D, window) in ((8, 128, 2), (16, 64, 1)):
        c = new_cache(S=window + 2, B=1, H=H, L=1500, D=D)
        c.head = window
        for mode, plan in ((mw.MW_QUEUED_ISOLATED, (2, 6)), (mw.MW_QUEUED_CAUSAL, (2, 0))):
            ws = lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), 3, 1500, window)
            assert lib.mw_chunk_attn_cached_plan(ctypes.byref(c), 3, 1500, window, mode, ws, ctypes.byref(ns),
                                                 ctypes.byref(nw)) == mw.MW_OK
            assert (ns.value, nw.value) == plan
    c8 = _lib.mw_kvcache()
    assert lib.mw_kvcache_init_fp8(ctypes.byref(c8), A, A, 3, 1, 1, 300, 128, 0.02, 0.02) == mw.MW_OK
    c8.head = 1
    ws = lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c8), 3, 300, 1)
    assert lib.mw_chunk_attn_cached_plan(ctypes.byref(c8), 3, 300, 1, mw.MW_QUEUED_ISOLATED, ws, ctypes.byref(ns),
                                         ctypes.byref(nw)) == mw.MW_OK
    assert (ns.value, nw.value) == (4, 1)


@pytest.mark.parametrize("e4m3", [False, True])
def test_cached_split_plan_fits_the_workspace(e4m3):
    """Over a sweep of shapes and workspace budgets, the plan's partials fit the budget, a plan
    with whole tiles leaves at least one tile split, and the workspace-size query covers the plan
    of either visibility rule."""
    lib = mw.load()
    ns, nw = ctypes.c_int(), ctypes.c_int()
    for (B, H, L, D, live, nq, ql) in [(1, 16, 2640, 128, 6, 4, 2640), (2, 12, 600, 128, 12, 8, 600),
                                       (1, 8, 1500, 128, 2, 3, 1500), (1, 16, 2640, 128, 6, 1, 200),
                                       (1, 3, 500, 128, 4, 2, 333), (2, 6, 96, 64, 3, 3, 96)]:
        if e4m3 and D != 128:
            continue
        c = _lib.mw_kvcache()
        if e4m3:
            assert lib.mw_kvcache_init_fp8(ctypes.byref(c), A, A, live + 1, B, H, L, D, 0.02, 0.02) == mw.MW_OK
        else:
            assert lib.mw_kvcache_init(ctypes.byref(c), A, A, live + 1, B, H, L, D) == mw.MW_OK
        c.head = live
        need = lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), nq, ql, live)
        tq = nq * ql
        for mode in (mw.MW_QUEUED_CAUSAL, mw.MW_QUEUED_ISOLATED):
            for ws in (need, need // 2, need // 5, 1 << 20, 0):
                assert lib.mw_chunk_attn_cached_plan(ctypes.byref(c), nq, ql, live, mode, ws, ctypes.byref(ns),
                                                     ctypes.byref(nw)) == mw.MW_OK
                n_splits, n_whole = ns.value, nw.value
                assert n_splits >= 1 and n_whole >= 0
                if n_splits == 1:
                    assert n_whole == 0
                    continue
                # rows per tile of the configuration the launcher picks: 256, or for D = 128 cached
                # attention with few rows 64 (<= 64) / 128 (bf16 <= 512, e4m3 <= 128)
                if D != 128 or tq > (128 if e4m3 else 512):
                    bm = 256
                else:
                    bm = 64 if tq <= 64 else (128 if (tq <= 128 or not e4m3) else 256)
                nqt = -(-tq // bm)
                assert n_whole < nqt
                rows = min(tq, (nqt - n_whole) * bm)
                assert n_splits * B * H * rows * (D + 2) * 4 <= ws
                if ws == need:
                    assert n_splits * B * H * rows * (D + 2) * 4 <= need


def test_cached_split_plan_validation():
    lib = mw.load()
    c = new_cache(S=8, B=1, H=16, L=2640, D=128)
    c.head = 6
    ns, nw = ctypes.c_int(), ctypes.c_int()
    plan = lib.mw_chunk_attn_cached_plan
    assert plan(ctypes.byref(c), 1, 64, 6, 0, 0, None, ctypes.byref(nw)) == mw.MW_EINVAL
    assert plan(ctypes.byref(c), 0, 64, 6, 0, 0, ctypes.byref(ns), ctypes.byref(nw)) == mw.MW_EINVAL
    assert plan(ctypes.byref(c), 1, 64, 7, 0, 0, ctypes.byref(ns), ctypes.byref(nw)) == mw.MW_EINVAL
    assert plan(ctypes.byref(c), 1, 64, 6, 5, 0, ctypes.byref(ns), ctypes.byref(nw)) == mw.MW_EINVAL
    assert plan(None, 1, 64, 6, 0, 0, ctypes.byref(ns), ctypes.byref(nw)) == mw.MW_EINVAL


def test_sink_and_rope_validation():
    lib = mw.load()
    c = new_cache(S=4, D=128)
    assert (c.sink_len, c.k_sink) == (0, None)
    assert lib.mw_kvcache_set_sink(ctypes.byref(c), None, A, 5) == mw.MW_EINVAL
    assert lib.mw_kvcache_set_sink(ctypes.byref(c), A, U, 5) == mw.MW_EALIGN
    assert lib.mw_kvcache_set_sink(ctypes.byref(c), A, A, -1) == mw.MW_EINVAL
    assert lib.mw_kvcache_set_sink(ctypes.byref(c), A, A, 7) == mw.MW_OK and c.sink_len == 7
    assert lib.mw_kvcache_set_sink(ctypes.byref(c), None, None, 0) == mw.MW_OK and c.sink_len == 0
    rope = lambda off, cnt, th=10000.0: ctypes.byref(_lib.mw_rope(off, cnt, th))
    shift = lib.mw_kvcache_rope_shift
    assert shift(ctypes.byref(c), 3, None, None) == mw.MW_EINVAL
    assert shift(ctypes.byref(c), 3, rope(1, 8), None) == mw.MW_EINVAL          # odd offset
    assert shift(ctypes.byref(c), 3, rope(0, 7), None) == mw.MW_EINVAL          # odd count
    assert shift(ctypes.byref(c), 3, rope(120, 16), None) == mw.MW_EINVAL       # past D
    assert shift(ctypes.byref(c), 3, rope(0, 130), None) == mw.MW_EINVAL        # more than 64 pairs
    assert shift(ctypes.byref(c), 3, rope(0, 44, 0.0), None) == mw.MW_EINVAL    # theta
    # nothing live or shift 0: valid, no device work
    assert shift(ctypes.byref(c), 3, rope(0, 44), None) == mw.MW_OK
    c.head = 2
    assert shift(ctypes.byref(c), 0, rope(0, 44), None) == mw.MW_OK


def test_snapshot_restore_descriptor():
    """The descriptor is plain data: copying it snapshots the ring, copying it back restores it."""
    lib = mw.load()
    c = new_cache(S=5)
    c.head = 4
    lib.mw_kvcache_evict(ctypes.byref(c), 2)
    snap = _lib.mw_kvcache.from_buffer_copy(c)
    c.head += 3
    lib.mw_kvcache_evict(ctypes.byref(c), 3)
    ctypes.memmove(ctypes.byref(c), ctypes.byref(snap), ctypes.sizeof(c))
    assert (c.head, c.tail) == (4, 2)
    assert [lib.mw_kvcache_slot_of(ctypes.byref(c), i) for i in range(6)] == [-1, -1, 2, 3, -1, -1]


def test_last_error_is_cleared_on_success():
    lib = mw.load()
    c = new_cache()
    lib.mw_kvcache_evict(ctypes.byref(c), 1)
    assert err()
    assert lib.mw_kvcache_evict(ctypes.byref(c), 0) == mw.MW_OK
    assert err() == ""


def test_missing_library_fails_loudly(tmp_path):
    saved = _lib._lib
    try:
        _lib._lib = None
        with pytest.raises(RuntimeError, match="not found"):
            _lib.load(str(tmp_path / "nope.so"))
    finally:
        _lib._lib = saved


def test_fp8_validation():
    """e4m3 cache, quantizer and fp8 attention reject bad arguments before any launch."""
    lib = mw.load()
    c = _lib.mw_kvcache()
    init8 = lib.mw_kvcache_init_fp8
    assert init8(None, A, A, 4, 1, 2, 16, 128, 1.0, 1.0) == mw.MW_EINVAL
    assert init8(ctypes.byref(c), A, A, 4, 1, 2, 16, 64, 1.0, 1.0) == mw.MW_EUNSUPPORTED
    assert init8(ctypes.byref(c), A, A, 4, 1, 2, 16, 128, 0.0, 1.0) == mw.MW_EINVAL
    assert init8(ctypes.byref(c), A, A, 4, 1, 2, 16, 128, 1.0, float("inf")) == mw.MW_EINVAL
    assert init8(ctypes.byref(c), A, U, 4, 1, 2, 16, 128, 1.0, 1.0) == mw.MW_EALIGN
    assert init8(ctypes.byref(c), A, A, 4, 1, 2, 16, 128, 0.5, 0.25) == mw.MW_OK
    assert (c.elem_bytes, c.k_scale, c.v_scale, c.D) == (1, 0.5, 0.25, 128)
    b = new_cache(S=4, B=1, H=2, L=16, D=128)
    assert (b.elem_bytes, b.k_scale, b.v_scale) == (2, 1.0, 1.0)
    rope = _lib.mw_rope(0, 44, 10000.0)
    c.head = 2
    assert lib.mw_kvcache_rope_shift(ctypes.byref(c), 3, ctypes.byref(rope), None) == mw.MW_OK  # recorded
    c.rope_total, c.rope_set = 0, 0
    cached = lambda cache, *a: lib.mw_chunk_attn_cached(A, A, A, 2, 16, ctypes.byref(cache), 1, 0, A, None, 0.125,
                                                        None, 0, None)
    assert cached(c) == mw.MW_EINVAL and "e4m3" in err()
    f8 = lambda cache, *a: lib.mw_chunk_attn_cached_fp8(*a[:3], 2, 16, ctypes.byref(cache), *a[3:], None, 0, None,
                                                        None)
    b.head = 2
    assert f8(b, A, A, A, 1, 0, A, None, 0.125, 1.0) == mw.MW_EINVAL and "bf16" in err()
    assert f8(c, A, A, A, 1, 0, A, None, 0.125, 0.0) == mw.MW_EINVAL and "q_scale" in err()
    assert f8(c, A, A, A, 1, 0, A, None, -1.0, 1.0) == mw.MW_EINVAL
    assert f8(c, None, A, A, 1, 0, A, None, 0.125, 1.0) == mw.MW_EINVAL
    assert f8(c, A, U, A, 1, 0, A, None, 0.125, 1.0) == mw.MW_EALIGN
    assert f8(c, A, A, A, 3, 0, A, None, 0.125, 1.0) == mw.MW_EINVAL and "window" in err()
    assert f8(c, A, A, A, 1, 5, A, None, 0.125, 1.0) == mw.MW_EINVAL
    assert lib.mw_chunk_attn_cached_fp8(A, A, A, 2, 16, ctypes.byref(c), 1, 0, A, None, 0.125, 1.0, None, 0,
                                        strides((0, 0, 128)), None) == mw.MW_EINVAL  # overlapping output view
    c.elem_bytes = 3                                                    # a corrupt descriptor
    assert f8(c, A, A, A, 1, 0, A, None, 0.125, 1.0) == mw.MW_EINVAL and "corrupt" in err()
    q = lib.mw_quantize_fp8
    assert q(None, None, A, 1, 2, 16, 128, 1.0, None) == mw.MW_EINVAL
    assert q(A, None, U, 1, 2, 16, 128, 1.0, None) == mw.MW_EALIGN
    assert q(A, None, A, 1, 2, 16, 96, 1.0, None) == mw.MW_EUNSUPPORTED
    assert q(A, None, A, 0, 2, 16, 128, 1.0, None) == mw.MW_EINVAL
    assert q(A, None, A, 1, 2, 16, 128, 0.0, None) == mw.MW_EINVAL
    assert q(A, None, A, 1, 2, 16, 128, 1e-39, None) == mw.MW_EINVAL   # 1 / scale overflows fp32
    assert q(A, strides((2 * 16 * 128, 16 * 128, 100)), A, 1, 2, 16, 128, 1.0, None) == mw.MW_EINVAL


def test_fp8_workspace_size_policy():
    """An e4m3 cache's workspace size covers the split partials and the window's keys rotated
    on load (always included, whether shifts are pending or not)."""
    lib = mw.load()
    c = _lib.mw_kvcache()
    assert lib.mw_kvcache_init_fp8(ctypes.byref(c), A, A, 8, 1, 16, 2640, 128, 0.02, 0.02) == mw.MW_OK
    c.head = 6
    kwin = 6 * 16 * 2640 * 128  # a multiple of 256
    small = lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), 1, 128, 6) - kwin
    assert small % (16 * 128 * 130 * 4) == 0 and small // (16 * 128 * 130 * 4) >= 8
    assert lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), 1, 128, 2) - 2 * 16 * 2640 * 128 >= 0


def test_fp8_reshift_record_and_pending_workspace():
    """e4m3 re-shift by rotation on load, host side: a shift only adds to rope_total and fixes
    the band; a later shift with another band or theta is rejected; S beyond MW_MAX_SLOTS is
    refused at init; with shifts pending the split plan gets the workspace left after the
    rotated window keys, and a call whose workspace cannot hold them fails before any launch."""
    lib = mw.load()
    c = _lib.mw_kvcache()
    assert lib.mw_kvcache_init_fp8(ctypes.byref(c), A, A, _lib.MW_MAX_SLOTS + 1, 1, 2, 16, 128, 1.0, 1.0) \
        == mw.MW_EUNSUPPORTED
    assert lib.mw_kvcache_init_fp8(ctypes.byref(c), A, A, 4, 1, 16, 2640, 128, 0.02, 0.02) == mw.MW_OK
    assert (c.rope_total, c.rope_set) == (0, 0) and list(c.rope_at_commit[:4]) == [0, 0, 0, 0]
    c.head, c.tail = 3, 0                                 # chunks 0, 1, 2 committed before any shift
    shift = lib.mw_kvcache_rope_shift
    assert shift(ctypes.byref(c), 3, ctypes.byref(_lib.mw_rope(0, 44, 10000.0)), None) == mw.MW_OK
    assert shift(ctypes.byref(c), -1, ctypes.byref(_lib.mw_rope(0, 44, 10000.0)), None) == mw.MW_OK
    assert (c.rope_total, c.rope_set, c.rope_offset, c.rope_count) == (2, 1, 0, 44)
    assert shift(ctypes.byref(c), 3, ctypes.byref(_lib.mw_rope(2, 44, 10000.0)), None) == mw.MW_EINVAL
    assert "band" in err()
    assert shift(ctypes.byref(c), 3, ctypes.byref(_lib.mw_rope(0, 44, 500.0)), None) == mw.MW_EINVAL
    assert shift(ctypes.byref(c), 3, ctypes.byref(_lib.mw_rope(1, 44, 10000.0)), None) == mw.MW_EINVAL
    assert c.rope_total == 2
    kwin = 3 * 16 * 2640 * 128
    need = lib.mw_chunk_attn_cached_workspace_size(ctypes.byref(c), 1, 64, 3)
    ns, nw = ctypes.c_int(0), ctypes.c_int(0)
    plan = lambda ws: (lib.mw_chunk_attn_cached_plan(ctypes.byref(c), 1, 64, 3, 0, ws, ctypes.byref(ns),
                                                     ctypes.byref(nw)), ns.value)
    assert plan(need) == (mw.MW_OK, plan(need - kwin + kwin)[1])
    splits_pending = plan(need)[1]
    assert plan(kwin)[1] == 1                             # nothing left for partials: unsplit
    c.rope_at_commit[0] = c.rope_at_commit[1] = c.rope_at_commit[2] = 2   # nothing pending
    assert plan(need - kwin)[1] == splits_pending         # the same partials fit without the rotated keys
    c.rope_at_commit[1] = 0                               # chunk 1 pending again
    f8 = lib.mw_chunk_attn_cached_fp8
    assert f8(A, A, A, 1, 64, ctypes.byref(c), 3, 0, A, None, 0.125, 1.0, A, kwin - 256, None, None) == mw.MW_EINVAL
    assert "rotated keys" in err()
    assert f8(A, A, A, 1, 64, ctypes.byref(c), 3, 0, A, None, 0.125, 1.0, None, 0, None, None) == mw.MW_EINVAL



def test_lse_output_checks():
    """The binding's check of a caller-supplied lse (cached calls, bf16 and e4m3, and the
    training forward) rejects a wrong dtype, shape, layout or device before any launch."""
    import torch
    shape = (1, 2, 6)
    dev = torch.device("cpu")
    _lib._check_lse(None, shape, dev)
    _lib._check_lse(torch.empty(shape, dtype=torch.float32), shape, dev)
    bad = [torch.empty(shape, dtype=torch.bfloat16),                    # wrong dtype
           torch.empty((1, 2), dtype=torch.float32),                     # [B,H]
           torch.empty((1, 2, 5), dtype=torch.float32),                  # too few rows
           torch.empty((1, 6, 2), dtype=torch.float32).transpose(1, 2)]  # not contiguous
    for t in bad:
        with pytest.raises(ValueError):
            _lib._check_lse(t, shape, dev)
    with pytest.raises(ValueError):
        _lib._check_lse(torch.empty(shape, dtype=torch.float32), shape, torch.device("meta"))

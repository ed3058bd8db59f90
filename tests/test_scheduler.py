"""The pipelined denoiser's plan (paper Sec. 3.5, Eq. 4, Eq. 6, Eq. 7): the oracle simulation
pinned against closed forms and the invariants the paper states, and the library's closed-form
planner (mw_sched_plan) checked against the simulation tick by tick.  Host only."""
import ctypes
import itertools
import math
from collections import deque

import pytest

import oracle
import paper_2608_01127_amd as mw

CONFIGS = [dict(window=w, stride=r, n_chunks=n, cache_chunks=c, frames_per_chunk=f, sink_frames=s, shift=sh,
                n_bins=nb)
           for (w, r) in [(1, 1), (4, 1), (8, 1), (8, 2), (7, 2), (6, 3), (5, 5), (64, 4)]
           for (n, c) in [(1, 0), (9, 3), (25, 6), (40, 24)]
           for (f, s) in [(2, 1), (3, 0)]
           for (sh, nb) in [(1.0, 0), (3.0, 0), (5.0, 50)]]


def sim(cfg):
    return oracle.simulate_pipeline(**cfg)


# ----------------------------------------------------------------------------- oracle pins

def test_shift_formula_identities():
    """Eq. 6 restated: s t / (1 + (s-1) t) = 1 / (1 + (1/t - 1) / s); fixed points 0 and 1;
    s = 1 is the identity; s > 1 moves every interior level up; monotone in t."""
    for s in (0.5, 1.0, 2.0, 3.0, 7.5):
        assert oracle.shifted_tau(0.0, s) == 0.0 and oracle.shifted_tau(1.0, s) == pytest.approx(1.0, abs=1e-15)
        prev = -1.0
        for i in range(1, 100):
            t = i / 100
            v = oracle.shifted_tau(t, s)
            assert v == pytest.approx(1.0 / (1.0 + (1.0 / t - 1.0) / s), rel=1e-13)
            assert v > prev
            prev = v
            if s == 1.0:
                assert v == pytest.approx(t, abs=1e-15)
            elif s > 1.0:
                assert v > t
            else:
                assert v < t


def test_unshifted_schedule_is_uniform():
    """s = 1, no bins: a chunk with U updates steps 1, 1 - 1/U, ..., 0 (Delta-tau = -1/U)."""
    for w, r in [(8, 1), (8, 2), (6, 3)]:
        U = w // r
        for p in sim(dict(window=w, stride=r, n_chunks=20, cache_chunks=4, frames_per_chunk=2)):
            for tau, dt in zip(p["tau"], p["dtau"]):
                assert dt == pytest.approx(-1.0 / U, abs=1e-15)
                assert tau * U == pytest.approx(round(tau * U), abs=1e-12)


@pytest.mark.parametrize("cfg", CONFIGS[::3], ids=lambda c: "w{window}r{stride}n{n_chunks}c{cache_chunks}".format(**c))
def test_schedule_invariants(cfg):
    """What the paper states, checked on the simulation: the window holds at most W chunks,
    older chunks are never noisier (Eq. 4), every update has Delta-tau <= 0 (Eq. 7), every
    chunk starts at tau = 1, follows its own updates and reaches tau = 0 exactly when it is
    committed, chunks commit once and in order, the cache is a FIFO of capacity C, and the
    re-shift is the evicted chunks' frames."""
    plans = sim(cfg)
    W, r, N, C, f = cfg["window"], cfg["stride"], cfg["n_chunks"], cfg["cache_chunks"], cfg["frames_per_chunk"]
    U = W // r
    assert len(plans) == (N - 1) // r + U
    state = {}          # chunk -> (last tick seen, tau after that tick)
    committed = []
    cache = deque()
    evicted = 0
    for t, p in enumerate(plans):
        assert p["tick"] == t and 1 <= p["n_active"] <= W and p["ids"] == list(range(p["first"], p["first"] + p["n_active"]))
        taus = p["tau"]
        assert all(a <= b for a, b in zip(taus, taus[1:]))                     # Eq. 4 (older = cleaner)
        assert p["pos_first"] == cfg["sink_frames"] + len(cache) * f
        for c, tau, dt in zip(p["ids"], taus, p["dtau"]):
            assert dt <= 0.0
            if c in state:
                last_t, tau_after = state[c]
                assert last_t == t - 1 and tau == pytest.approx(tau_after, abs=1e-15)  # consecutive updates
            else:
                assert tau == 1.0                                                # enters as pure noise
            state[c] = (t, tau + dt)
        for c in p["committed"]:
            assert state[c][1] == pytest.approx(0.0, abs=1e-15)                 # data endpoint at commit
            committed.append(c)
            cache.append(c)
        n_ev = 0
        while len(cache) > C:
            cache.popleft()
            n_ev += 1
        evicted += n_ev
        assert p["n_evict"] == n_ev and p["rope_shift"] == n_ev * f and p["cache_live"] == len(cache)
        if t >= U - 1 and (t + 1) * r <= N:
            assert p["n_active"] == U * r                                         # steady state
    assert committed == list(range(N))
    for c in range(N):                                                            # U updates each
        assert sum(c in p["ids"] for p in plans) == U


def test_binned_levels_are_multiples_of_the_bin():
    for p in sim(dict(window=8, stride=1, n_chunks=12, cache_chunks=3, frames_per_chunk=2, shift=3.0, n_bins=50)):
        for tau in p["tau"]:
            assert tau * 50 == pytest.approx(round(tau * 50), abs=1e-9)


# ----------------------------------------------------------------------------- library planner vs oracle

@pytest.mark.parametrize("cfg", CONFIGS, ids=lambda c: "w{window}r{stride}n{n_chunks}c{cache_chunks}f{frames_per_chunk}s{shift}b{n_bins}".format(**c))
def test_library_plan_matches_simulation(cfg):
    c = mw.sched_config(**cfg)
    plans = sim(cfg)
    assert mw.mw_sched_num_ticks(c) == len(plans)
    for t, p in enumerate(plans):
        q = mw.mw_sched_plan(c, t)
        for k in ("first", "n_active", "ids", "n_commit", "committed", "n_evict", "rope_shift", "cache_live",
                  "pos_first"):
            assert q[k] == p[k], (t, k)
        assert q["updates_per_chunk"] == cfg["window"] // cfg["stride"]
        for a, b in itertools.chain(zip(q["tau"], p["tau"]), zip(q["dtau"], p["dtau"])):
            assert a == pytest.approx(b, abs=1e-12)


def test_library_plan_validation():
    lib = mw.load()
    good = dict(window=8, stride=2, n_chunks=10, cache_chunks=4, frames_per_chunk=2, sink_frames=1, shift=3.0,
                n_bins=0)
    out = mw.mw_sched_tick()
    bad = [dict(window=0), dict(window=mw.MW_MAX_QUEUED + 1), dict(stride=0), dict(stride=9), dict(n_chunks=0),
           dict(cache_chunks=-1), dict(frames_per_chunk=0), dict(sink_frames=-1), dict(shift=0.0),
           dict(shift=float("inf")), dict(n_bins=-1)]
    for b in bad:
        cfg = mw.sched_config(**{**good, **b})
        assert lib.mw_sched_num_ticks(ctypes.byref(cfg)) == mw.MW_EINVAL, b
        assert lib.mw_sched_plan(ctypes.byref(cfg), 0, ctypes.byref(out)) == mw.MW_EINVAL, b
    cfg = mw.sched_config(**good)
    n = lib.mw_sched_num_ticks(ctypes.byref(cfg))
    assert n == (10 - 1) // 2 + 4
    assert lib.mw_sched_plan(ctypes.byref(cfg), n, ctypes.byref(out)) == mw.MW_EEMPTY
    assert lib.mw_sched_plan(ctypes.byref(cfg), -1, ctypes.byref(out)) == mw.MW_EEMPTY
    assert lib.mw_sched_plan(ctypes.byref(cfg), 0, None) == mw.MW_EINVAL
    assert lib.mw_sched_num_ticks(None) == mw.MW_EINVAL
    assert lib.mw_sched_plan(ctypes.byref(cfg), n - 1, ctypes.byref(out)) == mw.MW_OK
    assert out.n_active >= 1 and out.n_commit == out.n_active      # the last tick drains the window


def test_paper_shaped_plan():
    """The paper's streaming setting: 8 in-flight chunks, one new chunk per step, a 6- to
    24-chunk cache and a one-frame sink (Sec. 4.3): each chunk gets 8 updates, steady windows
    hold 8 chunks, and the cache never exceeds its capacity."""
    for C in (6, 12, 24):
        cfg = dict(window=8, stride=1, n_chunks=32, cache_chunks=C, frames_per_chunk=2, sink_frames=1, shift=3.0,
                   n_bins=0)
        plans = [mw.mw_sched_plan(mw.sched_config(**cfg), t) for t in range(mw.mw_sched_num_ticks(mw.sched_config(**cfg)))]
        assert all(p["updates_per_chunk"] == 8 for p in plans)
        assert max(p["n_active"] for p in plans) == 8 and max(p["cache_live"] for p in plans) == C
        assert sum(p["n_evict"] for p in plans) == 32 - C
        assert plans[-1]["cache_live"] == C and math.isclose(plans[7]["tau"][0], oracle.shifted_tau(1 / 8, 3.0))

"""Pipelined asynchronous denoising, simulated tick by tick (oracle; test infrastructure only).

Paper Sec. 3.5 ("Streaming Inference", "Structured Rolling KV Cache", "Pipelined
Denoising", and the latent update of Eq. 7) with the non-decreasing chunk
timesteps of Sec. 3.3 (Eq. 4) and the timestep shift of Sec. 3.4 (Eq. 6).

What the paper fixes: several future chunks are denoised at once inside an
active window, each at its own timestep; earlier chunks are never noisier than
later ones (Eq. 4); a chunk's latent moves by a step of size Delta-tau <= 0 per
update (Eq. 7); the sampler sizes Delta-tau so that every chunk reaches the
data endpoint (tau = 0) by the time it leaves the window, which depends on the
autoregressive stride and the window size; a finished chunk's keys and values
are committed to the FIFO cache, whose oldest chunks are evicted beyond its
capacity, after which the retained keys are re-indexed (RoPE re-shift) by the
evicted chunks' frames.

Reading taken where the paper gives no numbers:
- a tick is one DiT pass over the window; every in-flight chunk gets exactly one
  update per tick;
- ``stride`` new chunks (tau = 1) enter per tick, in order, while chunks remain;
  a chunk therefore stays U = floor(window / stride) ticks and gets U updates;
- before its k-th update (k = 0 .. U-1) a chunk is at tau = g(k / U) with
  g(x) = shift(1 - x), shift(t) = s t / (1 + (s - 1) t) (Eq. 6, applied to the
  inference grid as the experimental setup applies it to timesteps), so it starts at 1
  and its last update lands on g(1) = 0; with n_bins > 0 every level is rounded
  to the nearest multiple of 1 / n_bins (the discrete training-time bins);
- chunks that reach tau = 0 are committed in order after the tick, then the
  cache evicts its oldest chunks down to ``cache_chunks``; the re-shift is the
  evicted chunks' frames; the sink occupies the first ``sink_frames`` positions
  and is never evicted or shifted;
- positions are in frames of the re-indexed sequence [sink | cache | window].
"""
from __future__ import annotations

from collections import deque


def shifted_tau(t: float, s: float) -> float:
    """Timestep shift (Eq. 6): s t / (1 + (s - 1) t)."""
    return s * t / (1.0 + (s - 1.0) * t)


def tau_level(k: int, U: int, s: float, n_bins: int) -> float:
    """Noise level of a chunk before its k-th of U updates (k = U: after the last)."""
    tau = shifted_tau(1.0 - k / U, s)
    if n_bins > 0:
        tau = round(tau * n_bins) / n_bins
    return tau


def simulate(window: int, stride: int, n_chunks: int, cache_chunks: int, frames_per_chunk: int,
             sink_frames: int = 0, shift: float = 1.0, n_bins: int = 0) -> list:
    """Run the pipeline until every chunk is committed; one dict per tick.

    Each dict: tick, first (id of the oldest in-flight chunk), n_active, ids,
    tau (before this tick's update), dtau, n_commit, committed (ids), n_evict,
    rope_shift, cache_live (after the tick), pos_first (frame of the oldest
    in-flight chunk in the re-indexed sequence during the tick).
    """
    if not (window >= 1 and 1 <= stride <= window and n_chunks >= 1 and cache_chunks >= 0
            and frames_per_chunk >= 1 and sink_frames >= 0 and shift > 0 and n_bins >= 0):
        raise ValueError("invalid scheduler configuration")
    U = window // stride
    active = []                # [chunk id, updates done], oldest first
    cache = deque()            # committed chunk ids, oldest first
    next_id = 0
    committed_total = 0
    plans = []
    tick = 0
    while committed_total < n_chunks:
        for _ in range(stride):                       # admission of new noisy chunks
            if next_id < n_chunks:
                active.append([next_id, 0])
                next_id += 1
        assert 1 <= len(active) <= window
        ids = [c for c, _ in active]
        tau = [tau_level(k, U, shift, n_bins) for _, k in active]
        dtau = [tau_level(k + 1, U, shift, n_bins) - tau_level(k, U, shift, n_bins) for _, k in active]
        pos_first = sink_frames + len(cache) * frames_per_chunk
        for a in active:                              # one update each
            a[1] += 1
        done = [c for c, k in active if k == U]       # reached tau = 0
        active = [a for a in active if a[1] < U]
        for c in done:
            cache.append(c)
        committed_total += len(done)
        n_evict = 0
        while len(cache) > cache_chunks:
            cache.popleft()
            n_evict += 1
        plans.append({"tick": tick, "first": ids[0], "n_active": len(ids), "ids": ids, "tau": tau,
                      "dtau": dtau, "n_commit": len(done), "committed": done, "n_evict": n_evict,
                      "rope_shift": n_evict * frames_per_chunk, "cache_live": len(cache),
                      "pos_first": pos_first})
        tick += 1
    return plans

"""Plain fp64 block-causal attention (oracle; test infrastructure only).

Definitions followed
- Block-causal self-attention (paper Sec. 3.2): the token sequence is split
  into temporally ordered chunks; tokens of one chunk attend to each other in
  both directions, and a chunk attends to every token of the chunks before
  it, never to later chunks.  With chunks of ``chunk_len`` tokens aligned at
  token 0, token i lies in chunk floor(i / chunk_len) and query q may see key
  k iff chunk(k) <= chunk(q).  A shorter last chunk is allowed.
- Attention itself is the usual scaled dot-product softmax attention,
  O = softmax(s * Q K^T + M) V with M = 0 on visible and -inf on hidden
  pairs; s defaults to 1/sqrt(D).  LSE is the natural-log log-sum-exp of the
  masked, scaled logits of each row.
- The backward pass is the analytic softmax gradient:
  dV = P^T dO, dP = dO V^T, Delta = rowsum(dO * O), dS = P * (dP - Delta),
  dQ = s dS K, dK = s dS^T Q.
- Streaming visibility (paper Sec. 3.5): a chunk that is still being denoised
  sees the committed history and, under the chunk-wise causal constraint, the
  in-flight chunks that precede it in the active window (QUEUED_CAUSAL).  A
  stricter reading in which each in-flight chunk sees only the history and
  itself is provided as QUEUED_ISOLATED.

Everything is computed in float64 with numpy; no tiling, no skipping of
masked keys, no reordering beyond splitting query rows into blocks to bound
memory (rows are independent, so the split does not change any value).
"""
from __future__ import annotations

import numpy as np

QUEUED_CAUSAL = 0
QUEUED_ISOLATED = 1


def chunk_of(idx, chunk_len: int):
    """Chunk index of token positions ``idx`` (Sec. 3.2: chunks of chunk_len tokens from 0)."""
    return np.asarray(idx) // int(chunk_len)


def block_causal_visible(rows, n_keys: int, chunk_len: int) -> np.ndarray:
    """Boolean [len(rows), n_keys]: query row r may see key k iff chunk(k) <= chunk(r) (Sec. 3.2)."""
    rows = np.asarray(rows)
    keys = np.arange(n_keys)
    return chunk_of(keys, chunk_len)[None, :] <= chunk_of(rows, chunk_len)[:, None]


def attention_fwd(q, k, v, visible, scale):
    """Masked softmax attention for one head.

    q [R,D], k [N,D], v [N,Dv], visible bool [R,N] -> (O [R,Dv], LSE [R]) in fp64.
    Every row must have at least one visible key.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    s = scale * (q @ k.T)
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    l = e.sum(axis=1, keepdims=True)
    p = e / l
    o = p @ v
    lse = (m + np.log(l))[:, 0]
    return o, lse


def attention_bwd(q, k, v, do, visible, scale):
    """Analytic gradient of L = sum(dO * O) for one head; returns (dQ, dK, dV) in fp64."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    s = scale * (q @ k.T)
    s = np.where(visible, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    e = np.exp(s - m)
    p = e / e.sum(axis=1, keepdims=True)
    o = p @ v
    dv = p.T @ do
    dp = do @ v.T
    delta = (do * o).sum(axis=1, keepdims=True)
    ds = p * (dp - delta)
    dq = scale * (ds @ k)
    dk = scale * (ds.T @ q)
    return dq, dk, dv


def _default_scale(D, scale):
    return 1.0 / np.sqrt(D) if scale is None else float(scale)


def block_causal_attn_fwd(q, k, v, chunk_len: int, scale=None, row_block: int = 512):
    """Block-causal attention over [B,H,T,D] (Sec. 3.2).  Returns (O [B,H,T,D], LSE [B,H,T]).

    The mask is built explicitly for each block of query rows against all T
    keys; no key range is truncated.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, T, D = q.shape
    sc = _default_scale(D, scale)
    o = np.zeros((B, H, T, v.shape[-1]))
    lse = np.zeros((B, H, T))
    for r0 in range(0, T, row_block):
        rows = np.arange(r0, min(T, r0 + row_block))
        vis = block_causal_visible(rows, T, chunk_len)
        for b in range(B):
            for h in range(H):
                o[b, h, rows], lse[b, h, rows] = attention_fwd(q[b, h, rows], k[b, h], v[b, h], vis, sc)
    return o, lse


def block_causal_attn_fwd_rows(q, k, v, chunk_len: int, b: int, h: int, rows, scale=None):
    """Forward for selected query rows of one (b, h) only: (O [R,D], LSE [R])."""
    rows = np.asarray(rows)
    T, D = q.shape[2], q.shape[3]
    vis = block_causal_visible(rows, T, chunk_len)
    return attention_fwd(np.asarray(q[b, h, rows], np.float64), np.asarray(k[b, h], np.float64),
                         np.asarray(v[b, h], np.float64), vis, _default_scale(D, scale))


def block_causal_attn_bwd(q, k, v, do, chunk_len: int, scale=None, row_block: int = 512,
                          heads=None):
    """Gradients (dQ, dK, dV) of sum(dO * O) for block-causal attention over [B,H,T,D].

    Query rows are processed in blocks; dK and dV sum the contributions of all
    blocks.  ``heads`` optionally restricts the work to a list of (b, h)
    pairs (other heads' gradients are left at zero).
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    do = np.asarray(do, dtype=np.float64)
    B, H, T, D = q.shape
    sc = _default_scale(D, scale)
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    pairs = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    for r0 in range(0, T, row_block):
        rows = np.arange(r0, min(T, r0 + row_block))
        vis = block_causal_visible(rows, T, chunk_len)
        for b, h in pairs:
            # The row block's queries only; its contribution to dK/dV is additive.
            s = sc * (q[b, h, rows] @ k[b, h].T)
            s = np.where(vis, s, -np.inf)
            m = s.max(axis=1, keepdims=True)
            e = np.exp(s - m)
            p = e / e.sum(axis=1, keepdims=True)
            o = p @ v[b, h]
            dv[b, h] += p.T @ do[b, h, rows]
            dp = do[b, h, rows] @ v[b, h].T
            delta = (do[b, h, rows] * o).sum(axis=1, keepdims=True)
            ds = p * (dp - delta)
            dq[b, h, rows] = sc * (ds @ k[b, h])
            dk[b, h] += sc * (ds.T @ q[b, h, rows])
    return dq, dk, dv


def cached_visible(n_window: int, chunk_len, n_queued: int, q_len: int, mode: int) -> np.ndarray:
    """Visibility of the streaming step (Sec. 3.5) over the virtual key sequence.

    Keys are [committed history segments, oldest first] followed by [queued
    chunks 0..n_queued-1 (q_len tokens each)]; queries are the queued chunks.
    ``chunk_len`` is the length of every history segment (int) or a list of
    per-segment lengths (a sink segment first, then the window chunks).
    Virtual chunk ids: history segment i -> i, queued chunk j -> n_window + j.
    QUEUED_CAUSAL: key id <= query id (history plus preceding in-flight chunks).
    QUEUED_ISOLATED: key id < n_window or key id == query id.
    Returns bool [n_queued*q_len, sum(history lengths) + n_queued*q_len].
    """
    lens = [chunk_len] * n_window if np.isscalar(chunk_len) else list(chunk_len)
    assert len(lens) == n_window
    key_ids = np.concatenate([np.repeat(np.arange(n_window), lens).astype(int),
                              n_window + np.repeat(np.arange(n_queued), q_len)])
    q_ids = n_window + np.repeat(np.arange(n_queued), q_len)
    if mode == QUEUED_CAUSAL:
        return key_ids[None, :] <= q_ids[:, None]
    if mode == QUEUED_ISOLATED:
        return (key_ids[None, :] < n_window) | (key_ids[None, :] == q_ids[:, None])
    raise ValueError(f"unknown mode {mode}")


def cached_chunk_attn(q, k_new, v_new, window_k, window_v, n_queued: int, q_len: int,
                      mode: int = QUEUED_CAUSAL, scale=None, heads=None, sink_k=None, sink_v=None):
    """Attention of queued in-flight chunks over [sink || committed window || queued] (Sec. 3.5).

    q, k_new, v_new: [B,H,n_queued*q_len,D]; window_k/window_v: sequences of
    [B,H,chunk_len,D] arrays in logical order, oldest first (may be empty);
    sink_k/sink_v: optional [B,H,sink_len,D], the permanent sink anchor, placed
    first and visible to every queued chunk like the rest of the history.
    Returns (O [B,H,n_queued*q_len,D], LSE [B,H,n_queued*q_len]).
    """
    q = np.asarray(q, dtype=np.float64)
    B, H, NQ, D = q.shape
    assert NQ == n_queued * q_len
    hist_k = ([] if sink_k is None else [sink_k]) + list(window_k)
    hist_v = ([] if sink_v is None else [sink_v]) + list(window_v)
    lens = [np.asarray(c).shape[2] for c in hist_k]
    xk = np.concatenate([np.asarray(c, np.float64) for c in hist_k] + [np.asarray(k_new, np.float64)], axis=2)
    xv = np.concatenate([np.asarray(c, np.float64) for c in hist_v] + [np.asarray(v_new, np.float64)], axis=2)
    vis = cached_visible(len(hist_k), lens, n_queued, q_len, mode)
    sc = _default_scale(D, scale)
    o = np.zeros((B, H, NQ, xv.shape[-1]))
    lse = np.zeros((B, H, NQ))
    pairs = [(b, h) for b in range(B) for h in range(H)] if heads is None else list(heads)
    for b, h in pairs:
        o[b, h], lse[b, h] = attention_fwd(q[b, h], xk[b, h], xv[b, h], vis, sc)
    return o, lse


def rope_rotate(x, positions, dim_offset: int, dim_count: int, theta: float = 10000.0):
    """Rotary position embedding on one band of head dimensions (Sec. 3.5, RoPE re-shifting).

    Dimensions [dim_offset, dim_offset + dim_count) form dim_count/2 interleaved
    pairs (2i, 2i+1); pair i at position p is rotated by the angle
    p * theta^(-2i/dim_count).  Other dimensions are returned unchanged.
    x: [..., T, D]; positions: broadcastable to [..., T] (any real numbers).
    Re-shifting keys by -delta positions is rope_rotate(k, -delta, ...), since
    rotations by a and b compose to a rotation by a + b.
    """
    x = np.array(x, dtype=np.float64, copy=True)
    assert dim_count % 2 == 0 and dim_offset % 2 == 0 and dim_offset + dim_count <= x.shape[-1]
    npair = dim_count // 2
    freq = theta ** (-2.0 * np.arange(npair) / dim_count)
    ang = np.asarray(positions, dtype=np.float64)[..., None] * freq  # [..., T, npair]
    band = x[..., dim_offset:dim_offset + dim_count]
    a, b = band[..., 0::2].copy(), band[..., 1::2].copy()
    c, s = np.cos(ang), np.sin(ang)
    band[..., 0::2] = a * c - b * s
    band[..., 1::2] = a * s + b * c
    x[..., dim_offset:dim_offset + dim_count] = band
    return x

"""Pins for the fp64 oracle, independent of the oracle's own formulas.

Each test ties the oracle to something it does not share code with: a library
routine in a special case that reduces to it, a closed form, an invariant the
paper's definitions imply, finite differences, or brute force.
"""
import itertools

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from oracle import (QUEUED_CAUSAL, QUEUED_ISOLATED, RingError, RingModel,
                    block_causal_attn_bwd, block_causal_attn_fwd, cached_chunk_attn)

RNG = np.random.default_rng(7)


def rand(*shape, seed=0, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def kron_mask(T, L):
    """Block-causal mask built as a block lower-triangular matrix (independent construction)."""
    n = -(-T // L)
    blocks = np.kron(np.tril(np.ones((n, n))), np.ones((L, L)))
    return blocks[:T, :T].astype(bool)


def sdpa(q, k, v, mask=None, causal=False, scale=None):
    tq, tk, tv = (torch.tensor(x, dtype=torch.float64, requires_grad=True) for x in (q, k, v))
    m = None if mask is None else torch.tensor(mask)
    o = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=m, is_causal=causal,
                                                         scale=scale)
    return o, (tq, tk, tv)


def sdpa_grads(q, k, v, do, **kw):
    o, (tq, tk, tv) = sdpa(q, k, v, **kw)
    o.backward(torch.tensor(do))
    return o.detach().numpy(), tq.grad.numpy(), tk.grad.numpy(), tv.grad.numpy()


# ---------------------------------------------------------------- T1 / T2 / library mask

@pytest.mark.parametrize("B,H,T,D", [(1, 2, 48, 16), (2, 1, 37, 8)])
def test_single_chunk_is_bidirectional_attention(B, H, T, D):
    q, k, v, do = (rand(B, H, T, D, seed=s) for s in range(4))
    o, lse = block_causal_attn_fwd(q, k, v, chunk_len=T, row_block=16)
    ro, rdq, rdk, rdv = sdpa_grads(q, k, v, do)
    assert np.max(np.abs(o - ro)) < 1e-12
    dq, dk, dv = block_causal_attn_bwd(q, k, v, do, chunk_len=T, row_block=16)
    for a, b in ((dq, rdq), (dk, rdk), (dv, rdv)):
        assert np.max(np.abs(a - b)) < 1e-12
    # chunk_len larger than T is the same single chunk
    o2, _ = block_causal_attn_fwd(q, k, v, chunk_len=T + 5)
    assert np.array_equal(o2, o) or np.max(np.abs(o2 - o)) < 1e-15


@pytest.mark.parametrize("T,D", [(33, 8), (64, 16)])
def test_chunk_len_one_is_token_causal(T, D):
    q, k, v, do = (rand(1, 2, T, D, seed=10 + s) for s in range(4))
    o, _ = block_causal_attn_fwd(q, k, v, chunk_len=1, row_block=7)
    ro, rdq, rdk, rdv = sdpa_grads(q, k, v, do, causal=True)
    assert np.max(np.abs(o - ro)) < 1e-12
    dq, dk, dv = block_causal_attn_bwd(q, k, v, do, chunk_len=1, row_block=7)
    for a, b in ((dq, rdq), (dk, rdk), (dv, rdv)):
        assert np.max(np.abs(a - b)) < 1e-12


@pytest.mark.parametrize("T,L,D,scale", [(40, 8, 8, None), (45, 8, 16, None), (50, 7, 4, 0.37),
                                         (64, 64, 8, None), (30, 45, 8, None)])
def test_general_chunking_matches_library_masked_attention(T, L, D, scale):
    q, k, v, do = (rand(2, 3, T, D, seed=20 + s) for s in range(4))
    mask = kron_mask(T, L)
    o, lse = block_causal_attn_fwd(q, k, v, chunk_len=L, scale=scale, row_block=11)
    ro, rdq, rdk, rdv = sdpa_grads(q, k, v, do, mask=mask, scale=scale)
    assert np.max(np.abs(o - ro)) < 1e-12
    dq, dk, dv = block_causal_attn_bwd(q, k, v, do, chunk_len=L, scale=scale, row_block=11)
    for a, b in ((dq, rdq), (dk, rdk), (dv, rdv)):
        assert np.max(np.abs(a - b)) < 1e-12
    # LSE: library log-sum-exp over the visible logits only
    s = 1.0 / np.sqrt(D) if scale is None else scale
    for b_, h_ in ((0, 0), (1, 2)):
        logits = s * q[b_, h_] @ k[b_, h_].T
        for r in range(T):
            vis = mask[r]
            assert abs(lse[b_, h_, r] - scipy.special.logsumexp(logits[r, vis])) < 1e-12


def test_rows_function_matches_full():
    q, k, v = (rand(1, 2, 50, 8, seed=30 + s) for s in range(3))
    o, lse = block_causal_attn_fwd(q, k, v, chunk_len=12)
    rows = np.array([0, 11, 12, 30, 49])
    ro, rl = oracle.block_causal_attn_fwd_rows(q, k, v, 12, 0, 1, rows)
    assert np.max(np.abs(ro - o[0, 1, rows])) < 1e-14
    assert np.max(np.abs(rl - lse[0, 1, rows])) < 1e-14


def test_bwd_heads_subset():
    q, k, v, do = (rand(2, 2, 20, 4, seed=40 + s) for s in range(4))
    full = block_causal_attn_bwd(q, k, v, do, 6)
    part = block_causal_attn_bwd(q, k, v, do, 6, heads=[(1, 0)])
    for a, b in zip(full, part):
        assert np.array_equal(a[1, 0], b[1, 0])
        assert not b[0, 0].any()


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("T,L", [(24, 8), (26, 8), (5, 2)])
def test_zero_queries_average_visible_values(T, L):
    """Q = 0 makes every visible logit equal: O is the mean of the visible V rows, LSE = ln(#visible)."""
    D = 4
    q = np.zeros((1, 1, T, D))
    k = rand(1, 1, T, D, seed=1)
    v = rand(1, 1, T, D, seed=2)
    o, lse = block_causal_attn_fwd(q, k, v, chunk_len=L)
    for r in range(T):
        end = min(T, (r // L + 1) * L)
        assert np.max(np.abs(o[0, 0, r] - v[0, 0, :end].mean(axis=0))) < 1e-14
        assert abs(lse[0, 0, r] - np.log(end)) < 1e-14


def test_two_key_softmax_closed_form():
    """One query, two visible keys: O = sigmoid-weighted mix, a textbook closed form."""
    q = np.array([[[[1.0, 0.0]] * 3]])  # [1,1,3,2]
    k = np.array([[[[2.0, 0.0], [-1.0, 0.0], [50.0, 0.0]]]])
    v = np.array([[[[1.0, 0.0], [0.0, 1.0], [7.0, 7.0]]]])
    # chunk_len=2: rows 0,1 see keys 0,1 ; row 2 sees all
    o, lse = block_causal_attn_fwd(q, k, v, chunk_len=2, scale=1.0)
    w = 1.0 / (1.0 + np.exp(-3.0))  # weight of key 0 = e^2/(e^2+e^-1)
    assert np.max(np.abs(o[0, 0, 0] - np.array([w, 1 - w]))) < 1e-15
    assert abs(lse[0, 0, 1] - np.log(np.exp(2.0) + np.exp(-1.0))) < 1e-14


# ---------------------------------------------------------------- T3 invariants

def test_rows_sum_to_one_and_shift_invariances():
    B, H, T, D, L = 1, 2, 40, 8, 10
    q, k, v = (rand(B, H, T, D, seed=50 + s) for s in range(3))
    o1, _ = block_causal_attn_fwd(q, k, np.ones_like(v), chunk_len=L)
    assert np.max(np.abs(o1 - 1.0)) < 1e-12
    c = rand(D, seed=60)
    o, _ = block_causal_attn_fwd(q, k, v, chunk_len=L)
    ov, _ = block_causal_attn_fwd(q, k, v + c, chunk_len=L)
    assert np.max(np.abs(ov - (o + c))) < 1e-12
    ok_, _ = block_causal_attn_fwd(q, k + c, v, chunk_len=L)  # adds q.c to every logit of a row
    assert np.max(np.abs(ok_ - o)) < 1e-12


# ---------------------------------------------------------------- T4 permutation

def test_permutation_within_chunk_equivariant_and_across_chunks_not():
    B, H, T, D, L = 1, 1, 24, 4, 8
    q, k, v, do = (rand(B, H, T, D, seed=70 + s) for s in range(4))
    o, _ = block_causal_attn_fwd(q, k, v, chunk_len=L)
    g = block_causal_attn_bwd(q, k, v, do, chunk_len=L)
    perm = np.arange(T)
    for c in range(T // L):
        perm[c * L:(c + 1) * L] = c * L + np.random.default_rng(c).permutation(L)
    P = lambda x: x[:, :, perm]
    op, _ = block_causal_attn_fwd(P(q), P(k), P(v), chunk_len=L)
    assert np.max(np.abs(op - P(o))) < 1e-12
    gp = block_causal_attn_bwd(P(q), P(k), P(v), P(do), chunk_len=L)
    for a, b in zip(gp, g):
        assert np.max(np.abs(a - P(b))) < 1e-12
    # swapping a token across a chunk boundary must change the result (canary)
    cross = np.arange(T)
    cross[[L - 1, L]] = cross[[L, L - 1]]
    X = lambda x: x[:, :, cross]
    ox, _ = block_causal_attn_fwd(X(q), X(k), X(v), chunk_len=L)
    assert np.max(np.abs(ox - X(o))) > 1e-3


# ---------------------------------------------------------------- T6 finite differences

@pytest.mark.parametrize("T,L,D", [(7, 1, 3), (9, 3, 4), (10, 4, 2), (6, 6, 5), (11, 4, 8)])
def test_finite_difference_gradients(T, L, D):
    q, k, v, do = (rand(1, 1, T, D, seed=80 + s) for s in range(4))
    dq, dk, dv = block_causal_attn_bwd(q, k, v, do, chunk_len=L)
    h = 1e-6

    def loss(qq, kk, vv):
        o, _ = block_causal_attn_fwd(qq, kk, vv, chunk_len=L)
        return float((o * do).sum())

    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        num = np.zeros_like(x)
        for idx in itertools.product(*(range(n) for n in x.shape)):
            xp = x.copy(); xp[idx] += h
            xm = x.copy(); xm[idx] -= h
            args_p = {"q": q, "k": k, "v": v}; args_p[name] = xp
            args_m = {"q": q, "k": k, "v": v}; args_m[name] = xm
            num[idx] = (loss(args_p["q"], args_p["k"], args_p["v"]) -
                        loss(args_m["q"], args_m["k"], args_m["v"])) / (2 * h)
        rel = np.linalg.norm(num - g) / max(np.linalg.norm(g), 1e-30)
        assert rel < 1e-6, (name, rel)


# ---------------------------------------------------------------- T7 gradient identities

def test_gradient_sum_identities():
    B, H, T, D, L = 2, 2, 30, 8, 7
    q, k, v, do = (rand(B, H, T, D, seed=90 + s) for s in range(4))
    dq, dk, dv = block_causal_attn_bwd(q, k, v, do, chunk_len=L, row_block=9)
    # each softmax row's gradient sums to zero -> sum_k dK_k = 0
    assert np.max(np.abs(dk.sum(axis=2))) < 1e-12
    # each row's probabilities sum to one -> sum_k dV_k = sum_q dO_q
    assert np.max(np.abs(dv.sum(axis=2) - do.sum(axis=2))) < 1e-12


# ---------------------------------------------------------------- T8 causality, T9 chunk mass

def test_causality_exact():
    B, H, T, D, L = 1, 2, 40, 8, 10
    q, k, v, do = (rand(B, H, T, D, seed=100 + s) for s in range(4))
    o, lse = block_causal_attn_fwd(q, k, v, chunk_len=L)
    dq, _, _ = block_causal_attn_bwd(q, k, v, do, chunk_len=L)
    c = 2
    sl = slice(c * L, (c + 1) * L)
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[:, :, sl] += 3.0; k2[:, :, sl] -= 2.0; v2[:, :, sl] *= 5.0
    o2, lse2 = block_causal_attn_fwd(q2, k2, v2, chunk_len=L)
    dq2, _, _ = block_causal_attn_bwd(q2, k2, v2, do, chunk_len=L)
    assert np.array_equal(o2[:, :, :c * L], o[:, :, :c * L])
    assert np.array_equal(lse2[:, :, :c * L], lse[:, :, :c * L])
    assert np.array_equal(dq2[:, :, :c * L], dq[:, :, :c * L])
    assert not np.allclose(o2[:, :, c * L:], o[:, :, c * L:])


@pytest.mark.parametrize("T,L", [(40, 10), (43, 10)])
def test_chunk_mass_probe(T, L):
    n = -(-T // L)
    D = max(8, n)
    q, k = rand(1, 2, T, D, seed=110), rand(1, 2, T, D, seed=111)
    v = np.zeros((1, 2, T, D))
    v[:, :, np.arange(T), np.arange(T) // L] = 1.0
    o, _ = block_causal_attn_fwd(q, k, v, chunk_len=L)
    for r in range(T):
        c = r // L
        assert np.all(o[:, :, r, c + 1:] == 0.0)
        assert np.all(o[:, :, r, :c + 1] > 0.0)
        assert np.max(np.abs(o[:, :, r].sum(axis=-1) - 1.0)) < 1e-12


# ---------------------------------------------------------------- T5 cached attention

def _stream_case(B=1, H=2, L=6, D=8, n_hist=5, n_q=3, q_len=6, seed=120):
    hist_k = [rand(B, H, L, D, seed=seed + 2 * i) for i in range(n_hist)]
    hist_v = [rand(B, H, L, D, seed=seed + 2 * i + 1) for i in range(n_hist)]
    q = rand(B, H, n_q * q_len, D, seed=seed + 100)
    kn = rand(B, H, n_q * q_len, D, seed=seed + 101)
    vn = rand(B, H, n_q * q_len, D, seed=seed + 102)
    return hist_k, hist_v, q, kn, vn


def test_cached_full_history_equals_training_rows():
    """With every committed chunk in the window, paper-mode cached attention equals the
    block-causal forward over the whole sequence, restricted to the in-flight rows."""
    L = 6
    hk, hv, q, kn, vn = _stream_case(L=L, q_len=L)
    o, lse = cached_chunk_attn(q, kn, vn, hk, hv, n_queued=3, q_len=L, mode=QUEUED_CAUSAL)
    K = np.concatenate(hk + [kn], axis=2)
    V = np.concatenate(hv + [vn], axis=2)
    Qfull = np.concatenate([np.zeros_like(h) for h in hk] + [q], axis=2)
    of, lf = block_causal_attn_fwd(Qfull, K, V, chunk_len=L)
    n0 = len(hk) * L
    assert np.max(np.abs(o - of[:, :, n0:])) < 1e-12
    assert np.max(np.abs(lse - lf[:, :, n0:])) < 1e-12


def test_cached_window_equals_restricted_sequence():
    """A window of the newest w chunks equals full attention on the restricted sequence."""
    L = 6
    hk, hv, q, kn, vn = _stream_case(L=L, q_len=L)
    w = 2
    o, _ = cached_chunk_attn(q, kn, vn, hk[-w:], hv[-w:], n_queued=3, q_len=L)
    K = np.concatenate(hk[-w:] + [kn], axis=2)
    V = np.concatenate(hv[-w:] + [vn], axis=2)
    ro, _, _, _ = sdpa_grads(np.concatenate([np.zeros_like(hk[0])] * w + [q], axis=2), K, V,
                             np.zeros((1, 2, (w + 3) * L, 8)), mask=kron_mask((w + 3) * L, L))
    assert np.max(np.abs(o - ro[:, :, w * L:])) < 1e-12


def test_cached_isolated_mode():
    """Isolated mode: queued chunk j sees the window and itself only."""
    L, q_len, n_q = 6, 4, 3
    hk, hv, q, kn, vn = _stream_case(L=L, q_len=q_len, n_q=n_q)
    w = 3
    o, _ = cached_chunk_attn(q, kn, vn, hk[-w:], hv[-w:], n_queued=n_q, q_len=q_len,
                             mode=QUEUED_ISOLATED)
    for j in range(n_q):
        sl = slice(j * q_len, (j + 1) * q_len)
        K = np.concatenate(hk[-w:] + [kn[:, :, sl]], axis=2)
        V = np.concatenate(hv[-w:] + [vn[:, :, sl]], axis=2)
        ro, _ = sdpa(q[:, :, sl], K, V)
        assert np.max(np.abs(o[:, :, sl] - ro.detach().numpy())) < 1e-12


def test_cached_empty_window_and_mass_probe():
    L, q_len, n_q, w = 5, 3, 4, 2
    B, H, D = 1, 1, 8
    hk = [rand(B, H, L, D, seed=200 + i) for i in range(w)]
    q = rand(B, H, n_q * q_len, D, seed=210)
    kn = rand(B, H, n_q * q_len, D, seed=211)
    # values encode the virtual chunk id as one-hot
    hv = [np.zeros((B, H, L, D)) for _ in range(w)]
    for i in range(w):
        hv[i][..., i] = 1.0
    vn = np.zeros((B, H, n_q * q_len, D))
    for j in range(n_q):
        vn[:, :, j * q_len:(j + 1) * q_len, w + j] = 1.0
    for mode in (QUEUED_CAUSAL, QUEUED_ISOLATED):
        o, _ = cached_chunk_attn(q, kn, vn, hk, hv, n_queued=n_q, q_len=q_len, mode=mode)
        for j in range(n_q):
            rows = o[0, 0, j * q_len:(j + 1) * q_len]
            assert np.all(rows[:, w + j + 1:] == 0.0)
            if mode == QUEUED_ISOLATED:
                assert np.all(rows[:, w:w + j] == 0.0)
            assert np.max(np.abs(rows.sum(axis=1) - 1.0)) < 1e-12
    # empty window: causal mode is block-causal attention over the queued chunks alone
    o, _ = cached_chunk_attn(q, kn, vn, [], [], n_queued=n_q, q_len=q_len)
    of, _ = block_causal_attn_fwd(q, kn, vn, chunk_len=q_len)
    assert np.max(np.abs(o - of)) < 1e-12


# ---------------------------------------------------------------- ring model

def test_ring_model_against_brute_force_fifo():
    """Simulate slot storage and an explicit FIFO list; check for 300 steps that
    every live chunk is still stored in its slot and evicted chunks are gone."""
    S, W = 8, 6
    ring = RingModel(S)
    storage = [None] * S
    fifo = []
    rng = np.random.default_rng(3)
    nxt = 0
    for step in range(300):
        if ring.live < S and (rng.random() < 0.7 or ring.live == 0):
            slot = ring.append()
            storage[slot] = nxt
            fifo.append(nxt)
            nxt += 1
        else:
            n = int(rng.integers(0, ring.live + 1))
            ring.evict(n)
            fifo = fifo[n:]
        assert ring.live == len(fifo)
        for c in fifo:
            assert storage[ring.slot_of(c)] == c
        for c in range(nxt):
            if c not in fifo:
                assert ring.slot_of(c) == -1
        w = min(W, ring.live)
        assert ring.window(w) == fifo[len(fifo) - w:]


def test_ring_rollout_schedule_and_errors():
    S, W = 8, 6
    ring = RingModel(S)
    for t in range(200):
        slot = ring.append()
        assert slot == t % S
        if ring.live > W:
            ring.evict(ring.live - W)
        assert ring.live == min(t + 1, W)
        assert ring.window() == list(range(max(0, t + 1 - W), t + 1))
    r = RingModel(2)
    r.append(); r.append()
    with pytest.raises(RingError):
        r.append()
    with pytest.raises(RingError):
        r.evict(3)
    with pytest.raises(RingError):
        r.window(5)
    with pytest.raises(RingError):
        RingModel(0)


# ---------------------------------------------------------------- sink anchor and RoPE re-shift

def test_sink_is_history_visible_to_every_queued_chunk():
    """A sink segment behaves like one more (shorter) committed chunk placed first."""
    L, q_len, n_q = 6, 4, 3
    hk, hv, q, kn, vn = _stream_case(L=L, q_len=q_len, n_q=n_q)
    sk, sv = rand(1, 2, 3, 8, seed=300), rand(1, 2, 3, 8, seed=301)
    for mode in (QUEUED_CAUSAL, QUEUED_ISOLATED):
        o, _ = cached_chunk_attn(q, kn, vn, hk[-2:], hv[-2:], n_q, q_len, mode=mode, sink_k=sk, sink_v=sv)
        # reference: the isolated/causal rule over [sink, window] with an explicit boolean mask and SDPA
        K = np.concatenate([sk] + hk[-2:] + [kn], axis=2)
        V = np.concatenate([sv] + hv[-2:] + [vn], axis=2)
        nh = 3 + 2 * L
        mask = np.zeros((n_q * q_len, K.shape[2]), bool)
        for j in range(n_q):
            rows = slice(j * q_len, (j + 1) * q_len)
            mask[rows, :nh] = True
            lo = nh + (0 if mode == QUEUED_CAUSAL else j * q_len)
            mask[rows, lo:nh + (j + 1) * q_len] = True
        ro, _ = sdpa(q, K, V, mask=mask)
        assert np.max(np.abs(o - ro.detach().numpy())) < 1e-12


def test_rope_matches_complex_rotation():
    """Band rotation equals multiplying each interleaved pair, read as a complex number,
    by exp(i * p * theta^(-2k/n))."""
    x = rand(2, 5, 16, seed=310)
    pos = np.arange(5) * 1.5 - 2
    off, cnt, th = 4, 8, 500.0
    y = oracle.rope_rotate(x, pos, off, cnt, th)
    z = x[..., off:off + cnt:2] + 1j * x[..., off + 1:off + cnt:2]
    w = z * np.exp(1j * pos[:, None] * th ** (-np.arange(cnt // 2) * 2.0 / cnt))
    assert np.max(np.abs(y[..., off:off + cnt:2] - w.real)) < 1e-13
    assert np.max(np.abs(y[..., off + 1:off + cnt:2] - w.imag)) < 1e-13
    assert np.array_equal(y[..., :off], x[..., :off]) and np.array_equal(y[..., off + cnt:], x[..., off + cnt:])


def test_rope_group_properties_and_relative_positions():
    x = rand(3, 7, 12, seed=320)
    pa, pb = rand(3, 7, seed=321) * 5, rand(3, 7, seed=322) * 5
    r = lambda v, p: oracle.rope_rotate(v, p, 2, 8)
    assert np.max(np.abs(r(x, 0.0) - x)) < 1e-15
    assert np.max(np.abs(r(r(x, pa), pb) - r(x, pa + pb))) < 1e-12           # R(a) R(b) = R(a+b)
    assert np.max(np.abs(r(r(x, pa), -pa) - x)) < 1e-12                      # re-shift undoes a shift
    assert np.max(np.abs(np.linalg.norm(r(x, pa), axis=-1) - np.linalg.norm(x, axis=-1))) < 1e-12
    # q.k after rotation depends only on the position difference (what re-shifting preserves)
    q, k = rand(12, seed=323), rand(12, seed=324)
    d1 = r(q[None], np.array([9.0]))[0] @ r(k[None], np.array([4.0]))[0]
    d2 = r(q[None], np.array([5.0]))[0] @ r(k[None], np.array([0.0]))[0]
    assert abs(d1 - d2) < 1e-12

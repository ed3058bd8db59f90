"""GPU parity of block-causal attention forward/backward against the fp64 oracle (paper Sec. 3.2)."""
import numpy as np
import pytest

import oracle
import synth
from helpers import assert_close, bits_equal, f64, to_f64, to_gpu

pytestmark = pytest.mark.gpu


def run_fwd_bwd(mw, bits, L, with_bwd=True):
    q, k, v, do = (to_gpu(bits[n]) for n in ("q", "k", "v", "do"))
    o, lse = mw.mw_block_causal_attn_fwd(q, k, v, L)
    out = {"o": o, "lse": lse}
    if with_bwd:
        out["dq"], out["dk"], out["dv"] = mw.mw_block_causal_attn_bwd(q, k, v, o, do, lse, L)
    import torch
    torch.cuda.synchronize()
    return out


def small_case(B, H, T, D, L, seed):
    shp = (B, H, T, D)
    return {n: synth.normal_bf16(shp, seed + i) for i, n in enumerate(("q", "k", "v", "do"))}


# Sizes the oracle finishes in seconds, spanning several query/key tiles, ragged
# tails (T not a multiple of the tiles or of chunk_len) and the degenerate cases.
SMALL = [
    (1, 2, 256, 64, 64),     # the tiny configuration's shape
    (1, 2, 700, 64, 96),     # chunk edges inside tiles, ragged last chunk
    (2, 1, 1000, 128, 250),  # D=128, ragged tail
    (1, 1, 333, 64, 1),      # one token per chunk: token-causal
    (1, 1, 400, 128, 400),   # one chunk: bidirectional
    (1, 2, 130, 64, 1000),   # chunk longer than the sequence
    (1, 1, 1, 64, 1),        # single token
    (1, 1, 77, 128, 13),     # everything smaller than one tile
    (1, 2, 700, 72, 96),     # D=72 (the 0.5B model's head width): padded MFMA steps, ragged tail
    (2, 1, 300, 72, 300),    # D=72, one chunk
    (1, 1, 45, 72, 7),       # D=72, smaller than one tile
    # B*H a multiple of 8: the XCD work order that runs an XCD's heads' tiles
    # heaviest first across those heads, and (D = 64, 72) the one backward grid
    # whose dK/dV part is a multiple of 8 workgroups
    (2, 4, 700, 64, 96),     # chunk edges inside tiles, ragged last chunk
    (1, 8, 520, 72, 130),
    (2, 4, 300, 128, 100),
    # D = 128 (dK/dV work in 32-query steps with V staged in LDS): the degenerate chunkings
    (1, 1, 333, 128, 1),     # token-causal
    (1, 2, 130, 128, 1000),  # chunk longer than the sequence
    (1, 1, 1, 128, 1),       # single token
    (1, 2, 161, 128, 32),    # chunk edges on every 32-query step, ragged tail
]


@pytest.mark.parametrize("B,H,T,D,L", SMALL)
def test_small_fwd_bwd_vs_oracle(mw, B, H, T, D, L):
    print(f"[case] small B={B} H={H} T={T} D={D} L={L}", flush=True)
    bits = small_case(B, H, T, D, L, seed=1000 + T + D + L)
    g = run_fwd_bwd(mw, bits, L)
    q, k, v, do = (f64(bits[n]) for n in ("q", "k", "v", "do"))
    o, lse = oracle.block_causal_attn_fwd(q, k, v, L)
    assert_close("o", to_f64(g["o"]), o)
    assert_close("lse", to_f64(g["lse"]), lse, max_abs=2e-3, mean_abs=2e-4)
    dq, dk, dv = oracle.block_causal_attn_bwd(q, k, v, do, L)
    assert_close("dq", to_f64(g["dq"]), dq)
    assert_close("dk", to_f64(g["dk"]), dk)
    assert_close("dv", to_f64(g["dv"]), dv)


def test_tiny_config_fwd(mw):
    """B1 H2 D64, 4 chunks x 64 tokens, inputs drawn fp32 and rounded to bf16."""
    s = synth.TINY
    print(f"[case] {s.name}", flush=True)
    bits = synth.training_inputs(s)
    g = run_fwd_bwd(mw, bits, s.chunk_len, with_bwd=False)
    o, lse = oracle.block_causal_attn_fwd(f64(bits["q"]), f64(bits["k"]), f64(bits["v"]), s.chunk_len)
    assert_close("o", to_f64(g["o"]), o)
    assert_close("lse", to_f64(g["lse"]), lse, max_abs=2e-3, mean_abs=2e-4)


@pytest.fixture(scope="module")
def d64_run(mw):
    s = synth.TRAIN_D64
    print(f"[case] {s.name} (GPU fwd+bwd)", flush=True)
    bits = synth.training_inputs(s)
    g = run_fwd_bwd(mw, bits, s.chunk_len)
    return s, bits, {k: to_f64(v) for k, v in g.items()}


def test_train_d64_fwd_all_heads(d64_run):
    s, bits, g = d64_run
    o, lse = oracle.block_causal_attn_fwd(f64(bits["q"]), f64(bits["k"]), f64(bits["v"]), s.chunk_len)
    assert_close("o", g["o"], o)
    assert_close("lse", g["lse"], lse, max_abs=2e-3, mean_abs=2e-4)


@pytest.mark.parametrize("group", range(4))
def test_train_d64_bwd_heads(d64_run, group):
    """All 24 (b, h) heads in four groups of six."""
    s, bits, g = d64_run
    heads = [(b, h) for b in range(s.B) for h in range(s.H)][group * 6:(group + 1) * 6]
    q, k, v, do = (f64(bits[n]) for n in ("q", "k", "v", "do"))
    dq, dk, dv = oracle.block_causal_attn_bwd(q, k, v, do, s.chunk_len, heads=heads)
    idx = tuple(np.array(x) for x in zip(*heads))
    for name, ref in (("dq", dq), ("dk", dk), ("dv", dv)):
        assert_close(f"{name} heads {heads}", g[name][idx], ref[idx])


@pytest.fixture(scope="module")
def d128_run(mw):
    s = synth.TRAIN_D128
    print(f"[case] {s.name} (GPU fwd+bwd)", flush=True)
    bits = synth.training_inputs(s)
    g = run_fwd_bwd(mw, bits, s.chunk_len)
    return s, bits, g


@pytest.mark.parametrize("h", [0, 15])
def test_train_d128_head_vs_oracle(d128_run, h):
    """Full-length check of one head of the larger training shape (all rows, all gradients)."""
    s, bits, g = d128_run
    sel = lambda x: x[:, h:h + 1]
    q, k, v, do = (f64(sel(bits[n])) for n in ("q", "k", "v", "do"))
    o, lse = oracle.block_causal_attn_fwd(q, k, v, s.chunk_len, row_block=256)
    assert_close(f"o h{h}", to_f64(g["o"][:, h:h + 1]), o)
    assert_close(f"lse h{h}", to_f64(g["lse"][:, h:h + 1]), lse, max_abs=2e-3, mean_abs=2e-4)
    dq, dk, dv = oracle.block_causal_attn_bwd(q, k, v, do, s.chunk_len, row_block=256)
    for name, ref in (("dq", dq), ("dk", dk), ("dv", dv)):
        assert_close(f"{name} h{h}", to_f64(g[name][:, h:h + 1]), ref)


def test_train_d128_sampled_rows_all_heads(d128_run):
    """Every head, sampled query rows (including chunk edges and the last row), forward only."""
    s, bits, g = d128_run
    rows = np.array([0, 1, 2639, 2640, 5000, 21119, 21120, 39599, 39600, 42239])
    q, k, v = (f64(bits[n]) for n in ("q", "k", "v"))
    go, gl = to_f64(g["o"]), to_f64(g["lse"])
    for h in range(s.H):
        o, lse = oracle.block_causal_attn_fwd_rows(q, k, v, s.chunk_len, 0, h, rows)
        assert_close(f"o rows h{h}", go[0, h, rows], o)
        assert_close(f"lse rows h{h}", gl[0, h, rows], lse, max_abs=2e-3, mean_abs=2e-4)


# ------------------------------------------------------------------ exact-structure tests

def test_causality_bit_exact(mw):
    """Changing chunk c's Q/K/V leaves every output row of earlier chunks bit-identical."""
    import torch
    B, H, T, D, L = 1, 2, 900, 64, 200
    bits = small_case(B, H, T, D, L, seed=77)
    g1 = run_fwd_bwd(mw, bits, L)
    c = 2
    pert = {n: bits[n].copy() for n in bits}
    rng = np.random.default_rng(5)
    for n in ("q", "k", "v"):
        pert[n][:, :, c * L:(c + 1) * L] = synth.f32_to_bf16_bits(
            rng.standard_normal((B, H, L, D)).astype(np.float32) * 3)
    g2 = run_fwd_bwd(mw, pert, L)
    n0 = c * L
    for name in ("o", "dq"):
        assert bits_equal(g1[name][:, :, :n0].contiguous(), g2[name][:, :, :n0].contiguous()), name
    assert torch.equal(g1["lse"][:, :, :n0], g2["lse"][:, :, :n0])
    assert not torch.equal(g1["o"][:, :, n0:], g2["o"][:, :, n0:])


@pytest.mark.parametrize("T,D,L", [(1000, 64, 125), (1320, 128, 440)])
def test_chunk_mass_probe(mw, T, D, L):
    """V = one-hot(chunk of the key): the output's column c' is the softmax mass on chunk c';
    it must be exactly zero for every later chunk, and the masses sum to one."""
    import torch
    n = -(-T // L)
    bits = small_case(1, 2, T, D, L, seed=90 + D)
    v = np.zeros((1, 2, T, D), np.uint16)
    v[:, :, np.arange(T), np.arange(T) // L] = 0x3F80  # bf16 1.0
    bits["v"] = v
    g = run_fwd_bwd(mw, bits, L, with_bwd=False)
    o = to_f64(g["o"])
    for r in range(T):
        c = r // L
        assert np.all(o[:, :, r, c + 1:n] == 0.0), r
    assert np.max(np.abs(o.sum(axis=-1) - 1.0)) < 2e-2


def test_deterministic(mw):
    B, H, T, D, L = 1, 2, 1500, 128, 300
    bits = small_case(B, H, T, D, L, seed=55)
    g1 = run_fwd_bwd(mw, bits, L)
    g2 = run_fwd_bwd(mw, bits, L)
    for name in ("o", "dq", "dk", "dv"):
        assert bits_equal(g1[name], g2[name]), name

"""Pins of the E4M3 oracle (oracle/fp8.py) against the format's definition and an independent
implementation (torch's float8_e4m3fn conversion on the CPU), and of the fp8 attention reading:
attention on dequantized codes is plain attention, so the fp8 kernels are compared with
cached_chunk_attn on the dequantized values.  Host only."""
import numpy as np
import pytest

import oracle
import synth


def torch_e4m3(x):
    import torch
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def test_decode_table_from_the_definition():
    d = oracle.e4m3_decode
    assert d(0x00) == 0.0 and np.signbit(d(0x80)) and d(0x80) == 0.0
    assert d(0x01) == 2.0 ** -9 and d(0x07) == 7 * 2.0 ** -9          # subnormals m * 2^-9
    assert d(0x08) == 2.0 ** -6                                         # smallest normal
    assert d(0x38) == 1.0 and d(0x39) == 1.125 and d(0x40) == 2.0
    assert d(0x7E) == 448.0 and d(0xFE) == -448.0                        # largest finite
    assert np.isnan(d(0x7F)) and np.isnan(d(0xFF))                      # the only NaNs
    vals = d(np.arange(256))
    assert np.isfinite(vals).sum() == 254
    pos = vals[:0x7F]
    assert np.all(np.diff(pos) > 0)                                     # increasing with the code
    assert np.array_equal(vals[0x80:0xFF], -pos)                        # sign-magnitude


def test_decode_matches_torch_for_every_code():
    import torch
    t = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    mine = oracle.e4m3_decode(np.arange(256))
    fin = np.isfinite(mine)
    assert np.array_equal(np.isnan(t), ~fin) and np.array_equal(t[fin], mine[fin])


def test_encode_round_trips_every_finite_code():
    codes = np.array([c for c in range(256) if c not in (0x7F, 0xFF)], np.uint8)
    assert np.array_equal(oracle.e4m3_encode(oracle.e4m3_decode(codes)), codes)


def test_encode_ties_go_to_even_and_neighbours_to_the_nearest():
    pos = oracle.e4m3_decode(np.arange(0x7F))
    mids = (pos[1:] + pos[:-1]) / 2
    got = oracle.e4m3_encode(mids).astype(int)
    lo = np.arange(0x7E)
    assert np.array_equal(got, np.where(lo % 2 == 0, lo, lo + 1))
    below = np.nextafter(mids, 0)
    above = np.nextafter(mids, 1e9)
    assert np.array_equal(oracle.e4m3_encode(below).astype(int), lo)
    assert np.array_equal(oracle.e4m3_encode(above).astype(int), lo + 1)
    assert np.array_equal(oracle.e4m3_encode(-mids), got.astype(np.uint8) | 0x80)


def test_encode_matches_torch_on_random_values():
    rng = np.random.default_rng(11)
    x = np.concatenate([rng.standard_normal(20000) * 40, rng.standard_normal(5000) * 1e-2,
                        rng.uniform(-448, 448, 5000), rng.standard_normal(2000) * 1e-4]).astype(np.float32)
    assert np.array_equal(oracle.e4m3_encode(x), torch_e4m3(x))


def test_encode_rejects_out_of_range_and_quantize_saturates():
    with pytest.raises(ValueError):
        oracle.e4m3_encode([449.0])
    with pytest.raises(ValueError):
        oracle.e4m3_encode([np.nan])
    assert list(oracle.quantize_fp8(np.array([1e6, -1e6, 449.0, 448.0], np.float32), 1.0)) == [0x7E, 0xFE, 0x7E, 0x7E]


def test_quantize_is_exact_scaling_by_powers_of_two():
    rng = np.random.default_rng(3)
    x = synth.bf16_bits_to_f32(synth.normal_bf16((4096,), 77)).astype(np.float32)
    for k in (-3, 0, 5):
        s = 2.0 ** k
        assert np.array_equal(oracle.quantize_fp8(x, s), oracle.e4m3_encode(np.clip(x / np.float32(s), -448, 448)))
    # dequantized codes are within half an E4M3 step (relative 2^-4) of x / scale, or 2^-10 below 2^-6
    s = 0.0123
    q = oracle.dequantize_fp8(oracle.quantize_fp8(x, s), s) / np.float32(s)
    r = x / np.float64(np.float32(s))
    inr = np.abs(r) <= 448
    err = np.abs(q - r)[inr]
    bound = np.maximum(np.abs(r[inr]) * 2.0 ** -4, 2.0 ** -10) * (1 + 1e-6)
    assert np.all(err <= bound)


def test_quantize_uses_the_fp32_product():
    """fl32(x * fl32(1/s)) decides the code: a product that is not exactly representable in fp32 is
    rounded there first (checked against the same computation in fp32 by hand)."""
    x = np.array([1.0009765625, 3.0], np.float32)   # bf16 values
    s = np.float32(3.0)
    inv = np.float32(1.0) / s
    prod = x * inv
    assert prod.dtype == np.float32
    assert np.array_equal(oracle.quantize_fp8(x, 3.0), oracle.e4m3_encode(prod))


def test_fp8_attention_reading_is_attention_on_dequantized_values():
    """Cached attention on dequantized codes (the fp8 oracle) with per-tensor scales folded into
    q equals attention with the scale moved into the softmax scale (exactness of the reading)."""
    rng = np.random.default_rng(5)
    B, H, D, L, nq, qlen, W = 1, 1, 128, 16, 2, 16, 2
    codes = lambda shape: oracle.quantize_fp8(rng.standard_normal(shape).astype(np.float32), 0.02)
    q8, k8, v8 = (codes((B, H, nq * qlen, D)) for _ in range(3))
    wk = [codes((B, H, L, D)) for _ in range(W)]
    wv = [codes((B, H, L, D)) for _ in range(W)]
    deq = lambda c, s: oracle.dequantize_fp8(c, s)
    o1, l1 = oracle.cached_chunk_attn(deq(q8, 0.02), deq(k8, 0.02), deq(v8, 0.02), [deq(c, 0.02) for c in wk],
                                      [deq(c, 0.02) for c in wv], nq, qlen)
    s = float(np.float32(0.02))
    o2, l2 = oracle.cached_chunk_attn(oracle.e4m3_decode(q8), oracle.e4m3_decode(k8), oracle.e4m3_decode(v8),
                                      [oracle.e4m3_decode(c) for c in wk], [oracle.e4m3_decode(c) for c in wv], nq,
                                      qlen, scale=s * s / np.sqrt(D))
    np.testing.assert_allclose(o1, o2 * s, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l1, l2, rtol=1e-12, atol=1e-12)

"""The shared input generators: bf16 rounding agrees with torch's RNE cast, seeds are distinct."""
import numpy as np
import torch

import synth


def test_bf16_rounding_matches_torch():
    x = np.concatenate([synth.normal_f32((4096,), 5),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.0e38, -2.5e-39], np.float32)])
    bits = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, ref)
    back = synth.bf16_bits_to_f32(bits)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_seeds_distinct_and_reproducible():
    a = synth.training_inputs(synth.TINY)
    b = synth.training_inputs(synth.TINY)
    for k in a:
        assert np.array_equal(a[k], b[k])
    assert not np.array_equal(a["q"], a["k"])
    s0 = synth.stream_step_inputs(synth.STREAM, 0)
    s1 = synth.stream_step_inputs(synth.STREAM, 1, which=("q",))
    assert not np.array_equal(s0["q"], s1["q"])
    assert s0["k_commit"].shape == (1, 16, 2640, 128)
    assert s0["q"].shape == (1, 16, 4 * 2640, 128)

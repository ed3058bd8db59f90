"""Shared test utilities: moving synth's bf16 bit patterns to and from the GPU, and the parity bar."""
import numpy as np

import synth

# Binding tolerance for floating-point outputs vs the fp64 oracle (per tensor),
# on bf16-rounded inputs with fp32 accumulation on the GPU.
MAX_ABS = 2e-2
MEAN_ABS = 2e-3

# fp8 (e4m3) cached attention vs the fp64 oracle on the dequantized codes.  The
# kernel's only rounding beyond fp32 is that of the probabilities to e4m3
# before the PV product: a relative error of at most 2^-4 per weight (about
# 0.036 rms), so an output element moves by about 0.036 * sqrt(sum p^2 (v -
# o)^2) / sum p, which for unit-variance values over >= 64 visible keys is
# below 4e-3 on average and 2e-2 at the tails.  Bar: 2.5x the bf16 one.
FP8_MAX_ABS = 5e-2
FP8_MEAN_ABS = 5e-3


def to_gpu(bits, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def to_f64(t) -> np.ndarray:
    """bf16/fp32 torch tensor -> fp64 numpy (exact)."""
    import torch
    if t.dtype == torch.bfloat16:
        return synth.bf16_bits_to_f64(t.detach().cpu().view(torch.int16).numpy().view(np.uint16))
    return t.detach().cpu().double().numpy()


def f64(bits) -> np.ndarray:
    return synth.bf16_bits_to_f64(bits)


def assert_close(name, got, ref, max_abs=MAX_ABS, mean_abs=MEAN_ABS):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{name}: non-finite values"
    err = np.abs(got - ref)
    mx, mn = float(err.max()), float(err.mean())
    print(f"[parity] {name}: max_abs={mx:.3e} mean_abs={mn:.3e} (bar {max_abs:g}/{mean_abs:g})", flush=True)
    assert mx <= max_abs and mn <= mean_abs, f"{name}: max_abs={mx:.3e} mean_abs={mn:.3e}"
    return mx, mn


def bits_equal(a, b) -> bool:
    import torch
    return torch.equal(a.view(torch.int16), b.view(torch.int16))


def to_gpu_u8(codes, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(codes, dtype=np.uint8)).to(device)


def amax_scale(bits) -> float:
    """Per-tensor e4m3 scale that maps the tensor's largest magnitude to 448 (fp32)."""
    return float(np.float32(np.abs(synth.bf16_bits_to_f64(bits)).max() / 448.0))


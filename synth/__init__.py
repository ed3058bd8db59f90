"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This module only draws random numbers and rounds them to bfloat16; it holds
none of the attention arithmetic.  Both the fp64 oracle and the HIP path take
their inputs from here, so the two see bit-identical bf16 tensors.

Recipe (stands in for the VAE latents of the paper's DROID/RE10K videos,
which are not available): every tensor is drawn i.i.d. N(0, 1) in float32
from numpy's PCG64 generator with its own seed, then rounded to bfloat16
(round-to-nearest-even).  Layout is [B, H, T, D] with D innermost.
"""
from __future__ import annotations

import dataclasses

import numpy as np

# ---------------------------------------------------------------------------
# bf16 helpers (bit manipulation only)
# ---------------------------------------------------------------------------


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return uint16 bits.

    Inputs must be finite (the generators below only produce finite normals).
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return ((u >> 16) & 0xFFFF).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(bits).astype(np.float64)


def normal_f32(shape, seed: int) -> np.ndarray:
    """i.i.d. N(0,1) float32 from PCG64(seed)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return rng.standard_normal(size=shape, dtype=np.float32)


def normal_bf16(shape, seed: int) -> np.ndarray:
    """i.i.d. N(0,1) rounded to bfloat16; returns uint16 bit patterns."""
    return f32_to_bf16_bits(normal_f32(shape, seed))


# ---------------------------------------------------------------------------
# Workloads.  Shapes follow the latent-video chunking of the paper's method:
# a chunk is a few latent frames, each frame a grid of spatial tokens.
# ---------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class TrainShape:
    name: str
    B: int
    H: int
    T: int
    D: int
    chunk_len: int
    seed_base: int

    @property
    def n_chunks(self) -> int:
        return -(-self.T // self.chunk_len)


@dataclasses.dataclass(frozen=True)
class StreamShape:
    name: str
    B: int
    H: int
    D: int
    chunk_len: int      # tokens per committed chunk (ring slot length)
    n_queued: int       # in-flight chunks denoised together
    q_len: int          # tokens per queued chunk
    window: int         # committed chunks attended to
    slots: int          # ring capacity in chunks
    steps: int          # rollout length (chunk steps)
    seed_base: int
    sink_len: int = 0   # tokens of the sink anchor (0: none)


# tiny: 4 chunks x 64 tokens, two heads of width 64
TINY = TrainShape("tiny_fwd_B1H2T256D64L64", 1, 2, 256, 64, 64, 100000 * 1)
# training: 8 chunks x (3 latent frames x 440 tokens)
TRAIN_D64 = TrainShape("train_B2H12T10560D64L1320", 2, 12, 10560, 64, 1320, 100000 * 2)
# training, larger: 16 chunks x (3 frames x 880 tokens), head width 128
TRAIN_D128 = TrainShape("train_B1H16T42240D128L2640", 1, 16, 42240, 128, 2640, 100000 * 3)
# streaming: 4 in-flight chunks of 2640 tokens over 6 cached chunks in an 8-slot ring
STREAM = StreamShape("stream_B1H16D128L2640_nq4_W6_S8", 1, 16, 128, 2640, 4, 2640, 6, 8, 1,
                     100000 * 4)
# long rollout: 200 chunk steps of append + evict-to-window + cached attention
ROLLOUT = StreamShape("rollout_B1H16D128L2640_nq4_W6_S8_200steps", 1, 16, 128, 2640, 4, 2640,
                      6, 8, 200, 100000 * 5)

# The paper's own shapes (MiniWorld-1B: 12 heads of width 128; a chunk is 2
# latent frames of a 15 x 20 latent grid = 600 tokens; Sec. 4.1, Sec. 4.3):
# training over a 32-chunk window, and streaming with 8 in-flight chunks over a
# 24-chunk cache plus a one-frame (300-token) sink, with the classifier-free
# guidance batch of 2 (conditional and unconditional).
PAPER_1B_TRAIN = TrainShape("paper1b_train_B1H12T19200D128L600", 1, 12, 19200, 128, 600, 100000 * 6)
PAPER_1B_STREAM = StreamShape("paper1b_stream_B2H12D128L600_nq8_W24_S25_sink300", 2, 12, 128, 600, 8, 600, 24, 25,
                              1, 100000 * 7, sink_len=300)

TRAIN_SHAPES = {s.name: s for s in (TINY, TRAIN_D64, TRAIN_D128, PAPER_1B_TRAIN)}


def training_inputs(shape: TrainShape, which=("q", "k", "v", "do")) -> dict:
    """bf16 bit patterns for the training tensors, each [B,H,T,D].

    Seeds: seed_base + {q:0, k:1, v:2, do:3}; no two tensors share a seed.
    """
    offs = {"q": 0, "k": 1, "v": 2, "do": 3}
    shp = (shape.B, shape.H, shape.T, shape.D)
    return {name: normal_bf16(shp, shape.seed_base + offs[name]) for name in which}


def stream_step_inputs(shape: StreamShape, t: int, which=("k_commit", "v_commit", "q", "k_new", "v_new")) -> dict:
    """bf16 bit patterns for streaming step t.

    k_commit/v_commit: [B,H,chunk_len,D] (the chunk committed at step t);
    q/k_new/v_new: [B,H,n_queued*q_len,D] (the in-flight chunks).
    Seeds: seed_base + 10 + 8*t + {k_commit:0, v_commit:1, q:2, k_new:3, v_new:4}.
    """
    offs = {"k_commit": 0, "v_commit": 1, "q": 2, "k_new": 3, "v_new": 4}
    commit = (shape.B, shape.H, shape.chunk_len, shape.D)
    queued = (shape.B, shape.H, shape.n_queued * shape.q_len, shape.D)
    out = {}
    for name in which:
        shp = commit if name in ("k_commit", "v_commit") else queued
        out[name] = normal_bf16(shp, shape.seed_base + 10 + 8 * t + offs[name])
    return out


def random_bf16(shape, seed: int, scale: float = 1.0) -> np.ndarray:
    """Generic seeded N(0, scale^2) tensor as bf16 bits (small test cases)."""
    return f32_to_bf16_bits(normal_f32(shape, seed) * np.float32(scale))

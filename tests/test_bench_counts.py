"""The benchmark's useful-FLOP counts rest on its closed-form counts of visible (query, key) pairs:
check them against the oracle's explicit visibility masks (paper Sec. 3.2 block-causal, Sec. 3.5
queued chunks), and the headline figure of the D128 training shape against its closed form."""
import numpy as np
import pytest

import bench
import oracle
import synth


@pytest.mark.parametrize("T,L", [(256, 64), (700, 96), (333, 1), (400, 400), (130, 1000), (1000, 250), (77, 13)])
def test_block_causal_pairs_match_mask(T, L):
    vis = oracle.block_causal_visible(np.arange(T), T, L)
    assert bench.pairs_block_causal(2, 3, T, L) == 6 * int(vis.sum())


@pytest.mark.parametrize("mode", [oracle.QUEUED_CAUSAL, oracle.QUEUED_ISOLATED])
@pytest.mark.parametrize("w,L,nq,qlen", [(6, 40, 4, 40), (0, 32, 3, 17), (3, 50, 1, 64), (2, 25, 5, 25)])
def test_cached_pairs_match_mask(mode, w, L, nq, qlen):
    vis = oracle.cached_visible(w, L, nq, qlen, mode)
    causal = mode == oracle.QUEUED_CAUSAL
    assert bench.pairs_cached(1, 2, w, L, nq, qlen, causal=causal) == 2 * int(vis.sum())


def test_d128_training_pairs_closed_form():
    """16 chunks of 2640 tokens: chunk c sees c + 1 chunks, so P = B H L^2 * sum_c (c + 1) = 16 * 2640^2 * 136,
    and fwd + bwd useful FLOPs = 14 P D = 2.718e13."""
    s = synth.TRAIN_D128
    P = bench.pairs_block_causal(s.B, s.H, s.T, s.chunk_len)
    assert P == 16 * 2640 ** 2 * 136
    assert abs(14.0 * P * s.D - 2.718e13) / 2.718e13 < 1e-3


def test_bench_refuses_several_gpus():
    """One GPU only: --gpus above 1 exits with a message before touching a device."""
    import json
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode != 0
    assert "one GPU" in json.loads(r.stdout.strip().splitlines()[-1])["error"]

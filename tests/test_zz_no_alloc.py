"""The backward entry point that allocates nothing (mw_block_causal_attn_bwd_noalloc: its row
terms live in the library's own per-GPU scratch array) against the entry point that takes a
caller workspace, on the same inputs: two calls in a row, the second one smaller, so that it
runs on what the first left in the array."""
import numpy as np
import pytest

import oracle
import synth
from helpers import assert_close, bits_equal, f64, to_f64, to_gpu

pytestmark = pytest.mark.gpu


def _case(mw, B, H, T, D, L, seed):
    import torch
    print(f"[case] noalloc bwd B{B} H{H} T{T} D{D} L{L}", flush=True)
    bits = {n: synth.normal_bf16((B, H, T, D), seed + i) for i, n in enumerate(("q", "k", "v", "do"))}
    q, k, v, do = (to_gpu(bits[n]) for n in ("q", "k", "v", "do"))
    o, lse = mw.mw_block_causal_attn_fwd(q, k, v, L)
    ref = mw.mw_block_causal_attn_bwd(q, k, v, o, do, lse, L)
    got = tuple(torch.full_like(q, float("nan")) for _ in range(3))
    mw.mw_block_causal_attn_bwd_noalloc(q, k, v, o, do, lse, L, *got)
    torch.cuda.synchronize()
    return bits, ref, got


def test_noalloc_bwd_matches_workspace_entry(mw):
    for B, H, T, D, L, seed in ((2, 3, 1000, 128, 160, 7000), (1, 2, 300, 64, 64, 7100)):
        bits, ref, got = _case(mw, B, H, T, D, L, seed)
        for name, r, g in zip(("dq", "dk", "dv"), ref, got):
            # the same kernels on the same inputs: bit-identical
            assert bits_equal(r, g), f"{name} differs from the workspace entry point"
        # and within the parity bar of the oracle (last head)
        sel = lambda x: x[-1:, -1:]
        qf, kf, vf, dof = (f64(sel(bits[n])) for n in ("q", "k", "v", "do"))
        rdq, rdk, rdv = oracle.block_causal_attn_bwd(qf, kf, vf, dof, L)
        for name, g, r in zip(("dq", "dk", "dv"), got, (rdq, rdk, rdv)):
            assert_close(f"{name} (noalloc) B{B} H{H} T{T} D{D}", to_f64(g[-1:, -1:]), r)


def test_noalloc_bwd_rejects_rows_beyond_the_array(mw):
    """B*H*T above 4,194,304 rows is refused before anything is launched."""
    import torch
    B, H, T, D = 1, 1, 4194304 + 64, 64
    q = torch.empty((B, H, T, D), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((B, H, T), dtype=torch.float32, device="cuda")
    with pytest.raises(mw.MWError) as e:
        mw.mw_block_causal_attn_bwd_noalloc(q, q, q, q, q, lse, 64, q, q, q)
    assert e.value.code == mw.MW_EUNSUPPORTED
    torch.cuda.synchronize()

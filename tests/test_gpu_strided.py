"""GPU checks of the strided entry points: [B,T,H,D] and fused-QKV views are read and written in
place, with results bit-identical to the contiguous path (same arithmetic, other addresses) and
within the parity bar of the oracle."""
import numpy as np
import pytest

import oracle
import synth
from helpers import assert_close, bits_equal, f64, to_f64, to_gpu

pytestmark = pytest.mark.gpu


def sync():
    import torch
    torch.cuda.synchronize()


def fused_qkv(B, T, H, D, seed):
    """A [B,T,3,H,D] tensor (as a QKV projection writes it) and its q, k, v [B,H,T,D] views."""
    import torch
    bits = synth.normal_bf16((B, T, 3, H, D), seed)
    t = to_gpu(bits)
    return bits, t, t[:, :, 0].transpose(1, 2), t[:, :, 1].transpose(1, 2), t[:, :, 2].transpose(1, 2)


@pytest.mark.parametrize("B,H,T,D,L", [(2, 3, 300, 64, 96), (1, 2, 333, 128, 128), (1, 1, 70, 64, 70)])
def test_training_views_bit_identical_and_vs_oracle(mw, B, H, T, D, L):
    import torch
    print(f"[case] strided training B={B} H={H} T={T} D={D} L={L}", flush=True)
    bits, fused, q, k, v = fused_qkv(B, T, H, D, seed=4100 + T)
    assert not q.is_contiguous() and q.stride(-1) == 1
    do_bits = synth.normal_bf16((B, T, H, D), 4200 + T)
    do_bthd = to_gpu(do_bits)
    do = do_bthd.transpose(1, 2)                               # [B,H,T,D] view of a [B,T,H,D] tensor
    o_bthd = torch.empty((B, T, H, D), dtype=torch.bfloat16, device="cuda")
    o = o_bthd.transpose(1, 2)
    o, lse = mw.mw_block_causal_attn_fwd(q, k, v, L, out=o)
    grads = torch.empty((3, B, T, H, D), dtype=torch.bfloat16, device="cuda")
    dq, dk, dv = (grads[i].transpose(1, 2) for i in range(3))
    mw.mw_block_causal_attn_bwd(q, k, v, o, do, lse, L, dq=dq, dk=dk, dv=dv)
    # the contiguous path on copies of the same data
    qc, kc, vc, doc = (x.contiguous() for x in (q, k, v, do))
    o2, lse2 = mw.mw_block_causal_attn_fwd(qc, kc, vc, L)
    dq2, dk2, dv2 = mw.mw_block_causal_attn_bwd(qc, kc, vc, o2, doc, lse2, L)
    sync()
    assert bits_equal(o.contiguous(), o2) and bits_equal(lse, lse2)
    for a, b_ in ((dq, dq2), (dk, dk2), (dv, dv2)):
        assert bits_equal(a.contiguous(), b_)
    # and the oracle
    to_bhtd = lambda x: f64(np.ascontiguousarray(np.swapaxes(x, 1, 2)))
    qf, kf, vf = (to_bhtd(bits[:, :, i]) for i in range(3))
    ro, _ = oracle.block_causal_attn_fwd(qf, kf, vf, L)
    rdq, rdk, rdv = oracle.block_causal_attn_bwd(qf, kf, vf, to_bhtd(do_bits), L)
    assert_close("o", to_f64(o.contiguous()), ro)
    for n, a, r in (("dq", dq, rdq), ("dk", dk, rdk), ("dv", dv, rdv)):
        assert_close(n, to_f64(a.contiguous()), r)


@pytest.mark.parametrize("split", [True, False])
@pytest.mark.parametrize("D,nq,qlen", [(128, 2, 200), (128, 1, 64), (64, 3, 50)])
def test_cached_views_bit_identical(mw, split, D, nq, qlen):
    import torch
    B, H, L, S, W = 1, 2, 160, 4, 3
    print(f"[case] strided cached split={split} D={D} nq={nq} qlen={qlen}", flush=True)
    cache = mw.KVCache(S, B, H, L, D)
    chunks = [(synth.normal_bf16((B, L, H, D), 4300 + 2 * i), synth.normal_bf16((B, L, H, D), 4301 + 2 * i))
              for i in range(4)]
    ring = oracle.RingModel(S)
    for kc, vc in chunks:       # commit straight from [B,L,H,D] tensors
        kg, vg = to_gpu(kc).transpose(1, 2), to_gpu(vc).transpose(1, 2)
        slot = mw.mw_kvcache_append(cache, kg, vg)
        assert slot == ring.append()
        sync()
        assert bits_equal(cache.k_slots[slot], kg.contiguous()) and bits_equal(cache.v_slots[slot], vg.contiguous())
    Tq = nq * qlen
    bits, fused, q, k, v = fused_qkv(B, Tq, H, D, seed=4400 + Tq)
    o_bthd = torch.empty((B, Tq, H, D), dtype=torch.bfloat16, device="cuda")
    o, lse = mw.mw_chunk_attn_cached(q, k, v, nq, qlen, cache, window=W, out=o_bthd.transpose(1, 2),
                                     want_lse=True, split=split)
    o2, lse2 = mw.mw_chunk_attn_cached(q.contiguous(), k.contiguous(), v.contiguous(), nq, qlen, cache, window=W,
                                       want_lse=True, split=split)
    sync()
    assert bits_equal(o.contiguous(), o2) and bits_equal(lse, lse2)
    win = ring.window(W)
    to_bhtd = lambda x: f64(np.ascontiguousarray(np.swapaxes(x, 1, 2)))
    ro, _ = oracle.cached_chunk_attn(to_bhtd(bits[:, :, 0]), to_bhtd(bits[:, :, 1]), to_bhtd(bits[:, :, 2]),
                                     [to_bhtd(chunks[c][0]) for c in win], [to_bhtd(chunks[c][1]) for c in win],
                                     nq, qlen)
    assert_close("o", to_f64(o.contiguous()), ro)

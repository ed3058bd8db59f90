"""ctypes binding of libmw.so (include/mw.h).  Argument marshalling only.

Every function here forwards torch tensors' device pointers and the current
HIP stream to the C ABI; all arithmetic runs in the library's HIP kernels.
There is no fallback: if the library is missing or a call fails, an
exception is raised.
"""
from __future__ import annotations

import ctypes
import math
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmw.so")

MW_OK = 0
MW_EINVAL = -1
MW_EUNSUPPORTED = -2
MW_EALIGN = -3
MW_EFULL = -4
MW_EEMPTY = -5
MW_EHIP = -6
MW_QUEUED_CAUSAL = 0
MW_QUEUED_ISOLATED = 1
MW_MAX_WINDOW = 64
MW_MAX_QUEUED = 64
MW_MAX_SLOTS = 128

STATUS_NAMES = {0: "MW_OK", -1: "MW_EINVAL", -2: "MW_EUNSUPPORTED", -3: "MW_EALIGN", -4: "MW_EFULL",
                -5: "MW_EEMPTY", -6: "MW_EHIP"}


class MWError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(code, code)}: {msg}")
        self.code = code


class mw_kvcache(ctypes.Structure):
    _fields_ = [("k_slots", ctypes.c_void_p), ("v_slots", ctypes.c_void_p),
                ("S", ctypes.c_int), ("B", ctypes.c_int), ("H", ctypes.c_int), ("L", ctypes.c_int),
                ("D", ctypes.c_int), ("head", ctypes.c_int64), ("tail", ctypes.c_int64),
                ("k_sink", ctypes.c_void_p), ("v_sink", ctypes.c_void_p), ("sink_len", ctypes.c_int),
                ("elem_bytes", ctypes.c_int), ("k_scale", ctypes.c_float), ("v_scale", ctypes.c_float),
                ("rope_total", ctypes.c_int64), ("rope_offset", ctypes.c_int), ("rope_count", ctypes.c_int),
                ("rope_theta", ctypes.c_float), ("rope_set", ctypes.c_int),
                ("rope_at_commit", ctypes.c_int64 * MW_MAX_SLOTS)]


class mw_rope(ctypes.Structure):
    _fields_ = [("dim_offset", ctypes.c_int), ("dim_count", ctypes.c_int), ("theta", ctypes.c_float)]


class mw_strides(ctypes.Structure):
    _fields_ = [("b", ctypes.c_int64), ("h", ctypes.c_int64), ("t", ctypes.c_int64)]


class mw_sched_config(ctypes.Structure):
    _fields_ = [("window", ctypes.c_int), ("stride", ctypes.c_int), ("n_chunks", ctypes.c_int),
                ("cache_chunks", ctypes.c_int), ("frames_per_chunk", ctypes.c_int), ("sink_frames", ctypes.c_int),
                ("shift", ctypes.c_double), ("n_bins", ctypes.c_int)]


class mw_sched_tick(ctypes.Structure):
    _fields_ = [("tick", ctypes.c_int64), ("first", ctypes.c_int), ("n_active", ctypes.c_int),
                ("updates_per_chunk", ctypes.c_int),
                ("tau", ctypes.c_double * MW_MAX_QUEUED), ("dtau", ctypes.c_double * MW_MAX_QUEUED),
                ("n_commit", ctypes.c_int), ("n_evict", ctypes.c_int), ("rope_shift", ctypes.c_int),
                ("cache_live", ctypes.c_int), ("pos_first", ctypes.c_int)]


# Exported symbols and their signatures (mirrors include/mw.h).
_vp, _i, _f, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
_ip = ctypes.POINTER(ctypes.c_int)
_cache_p = ctypes.POINTER(mw_kvcache)
_str_p = ctypes.POINTER(mw_strides)
SIGNATURES = {
    "mw_last_error": ([], ctypes.c_char_p),
    "mw_version": ([], _i),
    "mw_block_causal_attn_fwd": ([_vp, _vp, _vp, _vp, _vp, _i, _i, _i, _i, _i, _f, _vp], _i),
    "mw_block_causal_attn_bwd_workspace_size": ([_i, _i, _i, _i], _sz),
    "mw_block_causal_attn_bwd": ([_vp] * 9 + [_vp, _sz, _i, _i, _i, _i, _i, _f, _vp], _i),
    "mw_kvcache_init": ([_cache_p, _vp, _vp, _i, _i, _i, _i, _i], _i),
    "mw_kvcache_append": ([_cache_p, _vp, _vp, _vp], _i),
    "mw_kvcache_evict": ([_cache_p, _i], _i),
    "mw_kvcache_set_sink": ([_cache_p, _vp, _vp, _i], _i),
    "mw_kvcache_rope_shift": ([_cache_p, _i, ctypes.POINTER(mw_rope), _vp], _i),
    "mw_kvcache_live": ([_cache_p], _i),
    "mw_kvcache_slot_of": ([_cache_p, ctypes.c_int64], _i),
    "mw_chunk_attn_cached_workspace_size": ([_cache_p, _i, _i, _i], _sz),
    "mw_chunk_attn_cached_plan": ([_cache_p, _i, _i, _i, _i, _sz, _ip, _ip], _i),
    "mw_chunk_attn_cached": ([_vp, _vp, _vp, _i, _i, _cache_p, _i, _i, _vp, _vp, _f, _vp, _sz, _vp], _i),
    "mw_block_causal_attn_fwd_strided": ([_vp, _vp, _vp, _vp, _vp, _str_p, _i, _i, _i, _i, _i, _f, _vp], _i),
    "mw_block_causal_attn_bwd_strided": ([_vp] * 9 + [_vp, _sz, _str_p, _i, _i, _i, _i, _i, _f, _vp], _i),
    "mw_block_causal_attn_bwd_noalloc": ([_vp] * 9 + [_i, _i, _i, _i, _i, _f, _vp], _i),
    "mw_kvcache_append_strided": ([_cache_p, _vp, _vp, _str_p, _vp], _i),
    "mw_chunk_attn_cached_strided": ([_vp, _vp, _vp, _i, _i, _cache_p, _i, _i, _vp, _vp, _f, _vp, _sz, _str_p,
                                      _vp], _i),
    "mw_quantize_fp8": ([_vp, _str_p, _vp, _i, _i, _i, _i, _f, _vp], _i),
    "mw_kvcache_init_fp8": ([_cache_p, _vp, _vp, _i, _i, _i, _i, _i, _f, _f], _i),
    "mw_chunk_attn_cached_fp8": ([_vp, _vp, _vp, _i, _i, _cache_p, _i, _i, _vp, _vp, _f, _f, _vp, _sz, _str_p, _vp],
                                 _i),
    "mw_sched_num_ticks": ([ctypes.POINTER(mw_sched_config)], ctypes.c_int64),
    "mw_sched_plan": ([ctypes.POINTER(mw_sched_config), ctypes.c_int64, ctypes.POINTER(mw_sched_tick)], _i),
}

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libmw.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libmw.so not found at {path}: build it with "
                           f"`python -m paper_2608_01127_amd.build` (no CPU fallback exists)")
    lib = ctypes.CDLL(path)
    for name, (args, res) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def _check(code: int) -> int:
    if code < 0:
        msg = load().mw_last_error().decode(errors="replace")
        raise MWError(code, msg)
    return code


# ----------------------------------------------------------------------------- torch glue

def _torch():
    import torch
    return torch


def _stream_handle(device) -> int:
    torch = _torch()
    return torch.cuda.current_stream(device).cuda_stream


def _ptr(t) -> int:
    return 0 if t is None else t.data_ptr()


def _bf16_4d(name, t, view: bool = False):
    """bf16 [B,H,T,D] on a GPU; contiguous, or (view=True) any view whose last
    dimension is contiguous (the library checks the remaining strides)."""
    torch = _torch()
    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16, got {t.dtype}")
    if t.dim() != 4:
        raise ValueError(f"{name} must be [B,H,T,D], got shape {tuple(t.shape)}")
    if view:
        if t.shape[-1] > 1 and t.stride(-1) != 1:
            raise ValueError(f"{name} must have a contiguous last (head) dimension")
    elif not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a GPU device")


def _u8_4d(name, t):
    """e4m3 codes as a contiguous uint8 [B,H,T,D] tensor on a GPU."""
    torch = _torch()
    if t.dtype != torch.uint8:
        raise TypeError(f"{name} must hold e4m3 codes as uint8, got {t.dtype}")
    if t.dim() != 4 or not t.is_contiguous() or t.device.type != "cuda":
        raise ValueError(f"{name} must be a contiguous [B,H,T,D] tensor on a GPU")


def _strides(*ts):
    """mw_strides array (B, H, T element strides) of the given [B,H,T,D] views."""
    arr = (mw_strides * len(ts))()
    for i, t in enumerate(ts):
        arr[i] = mw_strides(t.stride(0), t.stride(1), t.stride(2))
    return arr


def _check_lse(lse, shape, dev) -> None:
    """An lse output (or None): fp32, contiguous, of the given shape, on `dev`."""
    if lse is None:
        return
    torch = _torch()
    if lse.dtype != torch.float32 or tuple(lse.shape) != tuple(shape) or not lse.is_contiguous():
        raise ValueError(f"lse must be a contiguous fp32 tensor of shape {tuple(shape)}, got "
                         f"{lse.dtype} {tuple(lse.shape)}")
    if lse.device != dev:
        raise ValueError("lse must be on the device of the inputs")


def _same_device(*ts):
    dev = ts[0].device
    for t in ts:
        if t is not None and t.device != dev:
            raise ValueError("all tensors must be on the same device")
    return dev


def mw_block_causal_attn_fwd(q, k, v, chunk_len: int, scale=None, out=None, lse=None):
    """Block-causal attention forward.  q, k, v: bf16 [B,H,T,D] (views with a
    contiguous head dimension are read in place).  Returns (o, lse)."""
    torch = _torch()
    for n, t in (("q", q), ("k", k), ("v", v)):
        _bf16_4d(n, t, view=True)
    if k.shape != q.shape or v.shape != q.shape:
        raise ValueError("q, k, v must have the same shape")
    B, H, T, D = q.shape
    dev = _same_device(q, k, v)
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    o = torch.empty_like(q) if out is None else out
    lse = torch.empty((B, H, T), dtype=torch.float32, device=dev) if lse is None else lse
    _bf16_4d("out", o, view=True)
    if o.shape != q.shape:
        raise ValueError("out must have the shape of q")
    _same_device(q, o)
    _check_lse(lse, (B, H, T), dev)
    _check(load().mw_block_causal_attn_fwd_strided(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(lse),
                                                   _strides(q, k, v, o), B, H, T, D, int(chunk_len), scale,
                                                   _stream_handle(dev)))
    return o, lse


def mw_block_causal_attn_bwd_workspace_size(B: int, H: int, T: int, D: int) -> int:
    return int(load().mw_block_causal_attn_bwd_workspace_size(B, H, T, D))


def mw_block_causal_attn_bwd(q, k, v, o, d_o, lse, chunk_len: int, scale=None, workspace=None,
                             dq=None, dk=None, dv=None):
    """Backward of mw_block_causal_attn_fwd.  Returns (dq, dk, dv), bf16 [B,H,T,D]
    (views with a contiguous head dimension are accepted for every tensor)."""
    torch = _torch()
    for n, t in (("q", q), ("k", k), ("v", v), ("o", o), ("d_o", d_o)):
        _bf16_4d(n, t, view=True)
        if t.shape != q.shape:
            raise ValueError(f"{n} must have the shape of q")
    B, H, T, D = q.shape
    if lse.shape != (B, H, T) or lse.dtype != torch.float32 or not lse.is_contiguous():
        raise ValueError("lse must be fp32 [B,H,T] contiguous")
    dev = _same_device(q, k, v, o, d_o, lse)
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    need = mw_block_causal_attn_bwd_workspace_size(B, H, T, D)
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.empty_like(q) if dk is None else dk
    dv = torch.empty_like(q) if dv is None else dv
    for n, t in (("dq", dq), ("dk", dk), ("dv", dv)):
        _bf16_4d(n, t, view=True)
        if t.shape != q.shape:
            raise ValueError(f"{n} must have the shape of q")
    _same_device(q, workspace, dq, dk, dv)
    nbytes = workspace.numel() * workspace.element_size()
    _check(load().mw_block_causal_attn_bwd_strided(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(d_o), _ptr(lse),
                                                   _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), nbytes,
                                                   _strides(q, k, v, o, d_o, dq, dk, dv), B, H, T, D,
                                                   int(chunk_len), scale, _stream_handle(dev)))
    return dq, dk, dv


def mw_block_causal_attn_bwd_noalloc(q, k, v, o, d_o, lse, chunk_len: int, dq, dk, dv, scale=None):
    """The backward without a workspace: its row terms live in the library's own per-GPU
    scratch array, and neither the library nor this wrapper allocates anything, so dq, dk, dv
    must be given.  Contiguous bf16 [B,H,T,D] tensors, lse fp32 [B,H,T]; B*H*T <= 4,194,304.
    Calls that overlap on one GPU share the array and race.  Returns (dq, dk, dv)."""
    torch = _torch()
    for n, t in (("q", q), ("k", k), ("v", v), ("o", o), ("d_o", d_o), ("dq", dq), ("dk", dk), ("dv", dv)):
        _bf16_4d(n, t)
        if t.shape != q.shape:
            raise ValueError(f"{n} must have the shape of q")
    B, H, T, D = q.shape
    dev = _same_device(q, k, v, o, d_o, lse, dq, dk, dv)
    if lse is None:
        raise ValueError("lse is required")
    _check_lse(lse, (B, H, T), dev)
    scale = 1.0 / math.sqrt(D) if scale is None else float(scale)
    with torch.cuda.device(dev):  # the library takes the current device's copy of its array
        _check(load().mw_block_causal_attn_bwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(d_o), _ptr(lse),
                                                       _ptr(dq), _ptr(dk), _ptr(dv), B, H, T, D, int(chunk_len),
                                                       scale, _stream_handle(dev)))
    return dq, dk, dv


class KVCache:
    """Ring-buffered rolling KV cache over torch-owned slot tensors: bf16
    [S,B,H,L,D], or with fp8=True e4m3 codes (uint8 [S,B,H,L,D]) with the
    per-tensor scales k_scale, v_scale (value = code * scale).

    Wraps the mw_kvcache descriptor; `head`/`tail` count commits/evictions.
    """

    def __init__(self, S: int, B: int, H: int, L: int, D: int, device="cuda", k_slots=None, v_slots=None,
                 fp8: bool = False, k_scale: float = 1.0, v_scale: float = 1.0):
        torch = _torch()
        shape = (S, B, H, L, D)
        dt = torch.uint8 if fp8 else torch.bfloat16
        self.fp8 = bool(fp8)
        self.k_slots = torch.empty(shape, dtype=dt, device=device) if k_slots is None else k_slots
        self.v_slots = torch.empty(shape, dtype=dt, device=device) if v_slots is None else v_slots
        for n, t in (("k_slots", self.k_slots), ("v_slots", self.v_slots)):
            if t.shape != shape or t.dtype != dt or not t.is_contiguous():
                raise ValueError(f"{n} must be {dt} contiguous {shape}")
        self.desc = mw_kvcache()
        if fp8:
            _check(load().mw_kvcache_init_fp8(ctypes.byref(self.desc), _ptr(self.k_slots), _ptr(self.v_slots),
                                              S, B, H, L, D, float(k_scale), float(v_scale)))
        else:
            _check(load().mw_kvcache_init(ctypes.byref(self.desc), _ptr(self.k_slots), _ptr(self.v_slots),
                                          S, B, H, L, D))

    @property
    def head(self) -> int:
        return int(self.desc.head)

    @property
    def tail(self) -> int:
        return int(self.desc.tail)

    @property
    def live(self) -> int:
        return _check(load().mw_kvcache_live(ctypes.byref(self.desc)))

    def slot_of(self, chunk: int) -> int:
        return int(load().mw_kvcache_slot_of(ctypes.byref(self.desc), int(chunk)))

    def set_sink(self, k_sink, v_sink) -> None:
        """Keep k_sink/v_sink (bf16 [B,H,sink_len,D]) as the sink anchor; None removes it."""
        d = self.desc
        if k_sink is None:
            _check(load().mw_kvcache_set_sink(ctypes.byref(d), None, None, 0))
            self._sink = None
            return
        for n, t in (("k_sink", k_sink), ("v_sink", v_sink)):
            if self.fp8:
                _u8_4d(n, t)
            else:
                _bf16_4d(n, t)
            if tuple(t.shape[:2]) != (d.B, d.H) or t.shape[3] != d.D or t.shape != k_sink.shape:
                raise ValueError(f"{n} must be [B,H,sink_len,D] with B,H,D of the cache")
        _check(load().mw_kvcache_set_sink(ctypes.byref(d), _ptr(k_sink), _ptr(v_sink), int(k_sink.shape[2])))
        self._sink = (k_sink, v_sink)  # keep the tensors alive while the cache points at them

    def snapshot(self) -> bytes:
        """A copy of the whole descriptor (ring counters, sink, e4m3 re-shift record); the slot
        buffers' contents are the caller's to save alongside."""
        return bytes(self.desc)

    def restore(self, snap: bytes) -> None:
        ctypes.memmove(ctypes.byref(self.desc), snap, ctypes.sizeof(mw_kvcache))


def mw_kvcache_append(cache: KVCache, k_chunk, v_chunk) -> int:
    """Commit one chunk (bf16 [B,H,L,D], or a view of one with a contiguous head
    dimension); returns the slot it was written to."""
    d = cache.desc
    for n, t in (("k_chunk", k_chunk), ("v_chunk", v_chunk)):
        _bf16_4d(n, t, view=True)
        if tuple(t.shape) != (d.B, d.H, d.L, d.D):
            raise ValueError(f"{n} must be [B,H,L,D] = {(d.B, d.H, d.L, d.D)}")
    dev = _same_device(cache.k_slots, k_chunk, v_chunk)
    _check(load().mw_kvcache_append_strided(ctypes.byref(d), _ptr(k_chunk), _ptr(v_chunk),
                                            _strides(k_chunk, v_chunk), _stream_handle(dev)))
    # the slot the library wrote: the newest committed chunk's, by the library's own rule
    return _check(load().mw_kvcache_slot_of(ctypes.byref(d), int(d.head) - 1))


def mw_kvcache_evict(cache: KVCache, n_chunks: int) -> None:
    _check(load().mw_kvcache_evict(ctypes.byref(cache.desc), int(n_chunks)))


def mw_kvcache_set_sink(cache: KVCache, k_sink, v_sink) -> None:
    cache.set_sink(k_sink, v_sink)


def mw_kvcache_rope_shift(cache: KVCache, shift: int, dim_offset: int, dim_count: int, theta: float = 10000.0) -> None:
    """Rotate the keys of all live chunks by -shift positions on the rope band: in place for a
    bf16 cache; recorded, and applied when a call loads the window, for an e4m3 cache."""
    rope = mw_rope(int(dim_offset), int(dim_count), float(theta))
    _check(load().mw_kvcache_rope_shift(ctypes.byref(cache.desc), int(shift), ctypes.byref(rope),
                                        _stream_handle(cache.k_slots.device)))


def mw_kvcache_slot_of(cache: KVCache, chunk: int) -> int:
    return cache.slot_of(chunk)


def mw_chunk_attn_cached_workspace_size(cache: KVCache, n_queued: int, q_len: int, window: int = -1) -> int:
    return int(load().mw_chunk_attn_cached_workspace_size(ctypes.byref(cache.desc), int(n_queued), int(q_len),
                                                          int(window)))


def mw_chunk_attn_cached_plan(cache: KVCache, n_queued: int, q_len: int, window: int = -1,
                              flags: int = MW_QUEUED_CAUSAL, workspace_bytes: int = -1):
    """(n_splits, n_whole) the cached call uses with `workspace_bytes` of workspace
    (-1: the size mw_chunk_attn_cached_workspace_size gives)."""
    if workspace_bytes < 0:
        workspace_bytes = mw_chunk_attn_cached_workspace_size(cache, n_queued, q_len, window)
    ns, nw = ctypes.c_int(0), ctypes.c_int(0)
    _check(load().mw_chunk_attn_cached_plan(ctypes.byref(cache.desc), int(n_queued), int(q_len), int(window),
                                            int(flags), int(workspace_bytes), ctypes.byref(ns), ctypes.byref(nw)))
    return ns.value, nw.value


def mw_chunk_attn_cached(q, k_new, v_new, n_queued: int, q_len: int, cache: KVCache, window: int = -1,
                         flags: int = MW_QUEUED_CAUSAL, scale=None, out=None, lse=None, want_lse: bool = False,
                         workspace=None, split: bool = True):
    """Cached chunk attention of n_queued in-flight chunks.  Returns (o, lse or None).

    With split=True and no workspace given, a workspace of the size the library
    asks for is allocated here (torch); split=False runs the single-pass kernel.
    """
    torch = _torch()
    d = cache.desc
    for n, t in (("q", q), ("k_new", k_new), ("v_new", v_new)):
        _bf16_4d(n, t, view=True)
        if tuple(t.shape) != (d.B, d.H, n_queued * q_len, d.D):
            raise ValueError(f"{n} must be [B,H,n_queued*q_len,D] = {(d.B, d.H, n_queued * q_len, d.D)}")
    dev = _same_device(cache.k_slots, q, k_new, v_new)
    scale = 1.0 / math.sqrt(d.D) if scale is None else float(scale)
    o = torch.empty_like(q) if out is None else out
    _bf16_4d("out", o, view=True)
    if o.shape != q.shape:
        raise ValueError("out must have the shape of q")
    if want_lse and lse is None:
        lse = torch.empty((d.B, d.H, n_queued * q_len), dtype=torch.float32, device=dev)
    _check_lse(lse, (d.B, d.H, n_queued * q_len), dev)
    if split and workspace is None:
        need = mw_chunk_attn_cached_workspace_size(cache, n_queued, q_len, window)
        workspace = torch.empty(need, dtype=torch.uint8, device=dev) if need > 0 else None
    if not split:
        workspace = None
    _same_device(q, o, workspace)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().mw_chunk_attn_cached_strided(_ptr(q), _ptr(k_new), _ptr(v_new), int(n_queued), int(q_len),
                                               ctypes.byref(d), int(window), int(flags), _ptr(o), _ptr(lse), scale,
                                               _ptr(workspace), nbytes, _strides(q, k_new, v_new, o),
                                               _stream_handle(dev)))
    return o, lse


# ----------------------------------------------------------------------------- fp8 inference variant

def mw_quantize_fp8(x, scale: float, out=None):
    """bf16 [B,H,T,D] view -> contiguous e4m3 codes (uint8 [B,H,T,D]), code = RNE(clamp(x / scale))."""
    torch = _torch()
    _bf16_4d("x", x, view=True)
    B, H, T, D = x.shape
    y = torch.empty((B, H, T, D), dtype=torch.uint8, device=x.device) if out is None else out
    _u8_4d("out", y)
    if tuple(y.shape) != (B, H, T, D):
        raise ValueError("out must have the shape of x")
    _same_device(x, y)
    _check(load().mw_quantize_fp8(_ptr(x), _strides(x), _ptr(y), B, H, T, D, float(scale), _stream_handle(x.device)))
    return y


def mw_chunk_attn_cached_fp8(q8, k8_new, v8_new, n_queued: int, q_len: int, cache: KVCache, q_scale: float,
                             window: int = -1, flags: int = MW_QUEUED_CAUSAL, scale=None, out=None, lse=None,
                             want_lse: bool = False, workspace=None, split: bool = True):
    """Cached chunk attention over an e4m3 cache.  q8, k8_new, v8_new: e4m3 codes
    (uint8 [B,H,n_queued*q_len,D]; q8 with q_scale, k8/v8 with the cache's
    scales).  Returns (o bf16, lse or None)."""
    torch = _torch()
    d = cache.desc
    for n, t in (("q8", q8), ("k8_new", k8_new), ("v8_new", v8_new)):
        _u8_4d(n, t)
        if tuple(t.shape) != (d.B, d.H, n_queued * q_len, d.D):
            raise ValueError(f"{n} must be [B,H,n_queued*q_len,D] = {(d.B, d.H, n_queued * q_len, d.D)}")
    dev = _same_device(cache.k_slots, q8, k8_new, v8_new)
    scale = 1.0 / math.sqrt(d.D) if scale is None else float(scale)
    o = torch.empty(tuple(q8.shape), dtype=torch.bfloat16, device=dev) if out is None else out
    _bf16_4d("out", o, view=True)
    if o.shape != q8.shape:
        raise ValueError("out must have the shape of q8")
    if want_lse and lse is None:
        lse = torch.empty((d.B, d.H, n_queued * q_len), dtype=torch.float32, device=dev)
    _check_lse(lse, (d.B, d.H, n_queued * q_len), dev)
    if split and workspace is None:
        need = mw_chunk_attn_cached_workspace_size(cache, n_queued, q_len, window)
        workspace = torch.empty(need, dtype=torch.uint8, device=dev) if need > 0 else None
    if not split:
        workspace = None
    _same_device(q8, o, workspace)
    nbytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(load().mw_chunk_attn_cached_fp8(_ptr(q8), _ptr(k8_new), _ptr(v8_new), int(n_queued), int(q_len),
                                           ctypes.byref(d), int(window), int(flags), _ptr(o), _ptr(lse), scale,
                                           float(q_scale), _ptr(workspace), nbytes, _strides(o), _stream_handle(dev)))
    return o, lse


# ----------------------------------------------------------------------------- pipelined denoising schedule

def sched_config(window: int, stride: int, n_chunks: int, cache_chunks: int, frames_per_chunk: int,
                 sink_frames: int = 0, shift: float = 1.0, n_bins: int = 0) -> mw_sched_config:
    return mw_sched_config(int(window), int(stride), int(n_chunks), int(cache_chunks), int(frames_per_chunk),
                           int(sink_frames), float(shift), int(n_bins))


def mw_sched_num_ticks(cfg: mw_sched_config) -> int:
    return int(_check(load().mw_sched_num_ticks(ctypes.byref(cfg))))


def mw_sched_plan(cfg: mw_sched_config, tick: int) -> dict:
    """Plan of one tick of the pipelined denoiser (see include/mw.h) as a dict."""
    out = mw_sched_tick()
    _check(load().mw_sched_plan(ctypes.byref(cfg), int(tick), ctypes.byref(out)))
    n = out.n_active
    return {"tick": int(out.tick), "first": out.first, "n_active": n, "updates_per_chunk": out.updates_per_chunk,
            "ids": list(range(out.first, out.first + n)), "tau": list(out.tau[:n]), "dtau": list(out.dtau[:n]),
            "n_commit": out.n_commit, "committed": list(range(out.first, out.first + out.n_commit)),
            "n_evict": out.n_evict, "rope_shift": out.rope_shift, "cache_live": out.cache_live,
            "pos_first": out.pos_first}

"""ctypes binding of libmoba.so (C ABI in include/moba.h).

Argument marshalling only: torch tensors are described to the library as
(pointer, dtype, shape, strides) and the caller's current HIP stream is passed
through; every step of the computation runs in the library's HIP kernels.
There is no fallback: if libmoba.so is missing or fails to load, every call
raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmoba.so")

MOBA_F32, MOBA_BF16, MOBA_I32, MOBA_I64 = 0, 1, 2, 3
_DT = {torch.float32: MOBA_F32, torch.bfloat16: MOBA_BF16, torch.int32: MOBA_I32,
       torch.int64: MOBA_I64}

STATUS = ["MOBA_OK", "MOBA_ERR_NULL", "MOBA_ERR_DTYPE", "MOBA_ERR_SHAPE", "MOBA_ERR_LAYOUT",
          "MOBA_ERR_BLOCK_SIZE", "MOBA_ERR_TOPK", "MOBA_ERR_SEQLENS", "MOBA_ERR_UNSUPPORTED",
          "MOBA_ERR_NO_MEMORY", "MOBA_ERR_HIP"]


class MobaTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * 4), ("stride", ctypes.c_int64 * 4)]


class PhaseStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 24), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double)]


class MobaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        name = STATUS[status] if 0 <= status < len(STATUS) else str(status)
        super().__init__("%s failed: %s" % (fn, name))
        self.status = status
        self.name = name


_lib = None


def load() -> ctypes.CDLL:
    """Load libmoba.so once.  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError("libmoba.so not found at %s; build it with "
                           "`python -m paper_2502_13189_amd.build`" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(MobaTensor)
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    sig = {
        "moba_forward": [P, P, P, P, i32, i32, P, P, vp],
        "moba_backward": [P, P, P, P, i32, i32, P, P, P, P, P, P, vp],
        "moba_dense_backward": [P, P, P, P, P, P, P, P, P, P, vp],
        "moba_decode": [P, P, P, P, P, i32, i32, P, P, vp],
        "moba_decode_noalloc": [P, P, P, P, P, i32, i32, P, P, vp],
        "moba_dense_forward": [P, P, P, P, P, P, vp],
        "moba_pool": [P, P, i32, P, vp],
        "moba_select": [P, P, P, i32, i32, P, P, vp],
        "moba_route": [P, P, i32, i32, P, P, P, vp],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = ctypes.c_int
    i64 = ctypes.c_int64
    lib.moba_workspace_bytes.restype = ctypes.c_size_t
    lib.moba_workspace_bytes.argtypes = [i64, i32, i32, i32, i64, i32]
    lib.moba_workspace_held_bytes.restype = ctypes.c_size_t
    lib.moba_workspace_held_bytes.argtypes = []
    lib.moba_route_size.restype = ctypes.c_int
    lib.moba_route_size.argtypes = [P, i32, i32, i32, ctypes.POINTER(i64), ctypes.POINTER(i64), vp]
    lib.moba_take_wait_timeouts.restype = ctypes.c_int
    lib.moba_take_wait_timeouts.argtypes = [ctypes.POINTER(ctypes.c_uint64)]
    lib.moba_release_workspace.restype = ctypes.c_int
    lib.moba_release_workspace.argtypes = []
    lib.moba_status_string.restype = ctypes.c_char_p
    lib.moba_status_string.argtypes = [ctypes.c_int]
    lib.moba_profile_enable.argtypes = [ctypes.c_int]
    lib.moba_profile_enable.restype = None
    lib.moba_profile_read.argtypes = [ctypes.POINTER(PhaseStat), ctypes.c_int]
    lib.moba_profile_read.restype = ctypes.c_int
    _lib = lib
    return lib


def describe(t: torch.Tensor) -> MobaTensor:
    """Descriptor of a tensor (its storage stays owned by the caller)."""
    if t.dtype not in _DT:
        raise TypeError("unsupported dtype %s" % t.dtype)
    if t.dim() > 4:
        raise ValueError("at most 4 dimensions")
    d = MobaTensor()
    d.data = t.data_ptr()
    d.dtype = _DT[t.dtype]
    d.ndim = t.dim()
    for i in range(t.dim()):
        d.shape[i] = t.shape[i]
        d.stride[i] = t.stride(i)
    return d


def _ref(d):
    return None if d is None else ctypes.byref(d)


def _stream(t: torch.Tensor, stream=None) -> int:
    if stream is not None:
        return int(stream.cuda_stream if hasattr(stream, "cuda_stream") else stream)
    if t.is_cuda:
        return int(torch.cuda.current_stream(t.device).cuda_stream)
    return 0


def _check(fn: str, status: int):
    if status != 0:
        raise MobaError(fn, status)


def _cu(cu_seqlens) -> torch.Tensor:
    if not isinstance(cu_seqlens, torch.Tensor):
        cu_seqlens = torch.tensor(list(cu_seqlens), dtype=torch.int32)
    if cu_seqlens.dtype != torch.int32:
        cu_seqlens = cu_seqlens.to(torch.int32)
    return cu_seqlens.contiguous()


def forward(q, k, v, cu_seqlens, block_size: int, topk: int, out=None, lse=None, stream=None):
    """MoBA causal prefill forward.  q [T, Hq, 128], k/v [T, Hkv, 128] (bf16 or
    fp32, on the GPU); cu_seqlens [S+1] int32 (host tensor keeps the call
    asynchronous).  Returns (out [T, Hq, 128], lse [Hq, T] fp32)."""
    lib = load()
    cu = _cu(cu_seqlens)
    T, Hq = q.shape[0], q.shape[1]
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    if lse is None:
        lse = torch.empty((Hq, T), dtype=torch.float32, device=q.device)
    dq, dk, dv, dc, do, dl = map(describe, (q, k, v, cu, out, lse))
    _check("moba_forward", lib.moba_forward(_ref(dq), _ref(dk), _ref(dv), _ref(dc), int(block_size),
                                            int(topk), _ref(do), _ref(dl), _stream(q, stream)))
    return out, lse


def backward(q, k, v, cu_seqlens, block_size: int, topk: int, out, lse, dout, dq=None, dk=None,
             dv=None, stream=None):
    """Gradients of forward() w.r.t. q, k, v (bf16).  out and lse are forward()'s
    results for the same inputs; dout [T, Hq, 128] is the gradient w.r.t. out.
    Returns (dq [T, Hq, 128], dk [T, Hkv, 128], dv [T, Hkv, 128])."""
    lib = load()
    cu = _cu(cu_seqlens)
    if dq is None:
        dq = torch.empty_like(q, memory_format=torch.contiguous_format)
    if dk is None:
        dk = torch.empty_like(k, memory_format=torch.contiguous_format)
    if dv is None:
        dv = torch.empty_like(v, memory_format=torch.contiguous_format)
    d = [describe(t) for t in (q, k, v, cu, out, lse, dout, dq, dk, dv)]
    _check("moba_backward", lib.moba_backward(_ref(d[0]), _ref(d[1]), _ref(d[2]), _ref(d[3]),
                                              int(block_size), int(topk), _ref(d[4]), _ref(d[5]),
                                              _ref(d[6]), _ref(d[7]), _ref(d[8]), _ref(d[9]),
                                              _stream(q, stream)))
    return dq, dk, dv


def dense_backward(q, k, v, cu_seqlens, out, lse, dout, dq=None, dk=None, dv=None, stream=None):
    """Gradients of dense_forward() (causal full attention) w.r.t. q, k, v (bf16)."""
    lib = load()
    cu = _cu(cu_seqlens)
    if dq is None:
        dq = torch.empty_like(q, memory_format=torch.contiguous_format)
    if dk is None:
        dk = torch.empty_like(k, memory_format=torch.contiguous_format)
    if dv is None:
        dv = torch.empty_like(v, memory_format=torch.contiguous_format)
    d = [describe(t) for t in (q, k, v, cu, out, lse, dout, dq, dk, dv)]
    _check("moba_dense_backward", lib.moba_dense_backward(
        _ref(d[0]), _ref(d[1]), _ref(d[2]), _ref(d[3]), _ref(d[4]), _ref(d[5]), _ref(d[6]),
        _ref(d[7]), _ref(d[8]), _ref(d[9]), _stream(q, stream)))
    return dq, dk, dv


def decode(q, k_cache, v_cache, cu_seqlens, block_size: int, topk: int, kbar=None, out=None,
           lse=None, stream=None):
    """One new query per sequence against its cache (topk == 0: full
    attention).  q [S, Hq, 128] bf16; k_cache/v_cache [T, Hkv, 128] bf16 with
    each new token's key/value last in its sequence; kbar: optional block
    means from pool().  Returns (out [S, Hq, 128], lse [Hq, S])."""
    lib = load()
    cu = _cu(cu_seqlens)
    S, Hq = q.shape[0], q.shape[1]
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    if lse is None:
        lse = torch.empty((Hq, S), dtype=torch.float32, device=q.device)
    d = [describe(t) for t in (q, k_cache, v_cache, cu)]
    dkb = describe(kbar) if kbar is not None else None
    do, dl = describe(out), describe(lse)
    _check("moba_decode", lib.moba_decode(_ref(d[0]), _ref(d[1]), _ref(d[2]), _ref(d[3]),
                                          _ref(dkb), int(block_size), int(topk), _ref(do),
                                          _ref(dl), _stream(q, stream)))
    return out, lse


def decode_noalloc(q, k_cache, v_cache, cu_seqlens, block_size: int, topk: int, out, lse,
                   kbar=None, stream=None):
    """decode() through moba_decode_noalloc: the library allocates nothing;
    the caller passes out [S, Hq, 128] bf16 and lse [Hq, S] fp32, and
    cu_seqlens must be a host tensor."""
    lib = load()
    cu = _cu(cu_seqlens)
    d = [describe(t) for t in (q, k_cache, v_cache, cu)]
    dkb = describe(kbar) if kbar is not None else None
    do, dl = describe(out), describe(lse)
    _check("moba_decode_noalloc", lib.moba_decode_noalloc(_ref(d[0]), _ref(d[1]), _ref(d[2]),
                                                          _ref(d[3]), _ref(dkb), int(block_size),
                                                          int(topk), _ref(do), _ref(dl),
                                                          _stream(q, stream)))
    return out, lse


def dense_forward(q, k, v, cu_seqlens, out=None, lse=None, stream=None):
    """Dense causal attention with the same conventions as forward()."""
    lib = load()
    cu = _cu(cu_seqlens)
    T, Hq = q.shape[0], q.shape[1]
    if out is None:
        out = torch.empty_like(q, memory_format=torch.contiguous_format)
    if lse is None:
        lse = torch.empty((Hq, T), dtype=torch.float32, device=q.device)
    dq, dk, dv, dc, do, dl = map(describe, (q, k, v, cu, out, lse))
    _check("moba_dense_forward", lib.moba_dense_forward(_ref(dq), _ref(dk), _ref(dv), _ref(dc),
                                                        _ref(do), _ref(dl), _stream(q, stream)))
    return out, lse


def route_size(cu_seqlens, block_size: int, topk: int, num_q_heads: int, stream=None):
    """(nblk_total, E) as the library reports them: the batch's block count
    and its number of history selections (moba_route's entries)."""
    lib = load()
    cu = _cu(cu_seqlens)
    nb, e = ctypes.c_int64(), ctypes.c_int64()
    dc = describe(cu)
    _check("moba_route_size", lib.moba_route_size(_ref(dc), int(block_size), int(topk),
                                                  int(num_q_heads), ctypes.byref(nb),
                                                  ctypes.byref(e), _stream(cu, stream)))
    return int(nb.value), int(e.value)


def num_blocks(cu_seqlens, block_size: int) -> int:
    return route_size(cu_seqlens, block_size, 1, 1)[0]


def pool(k, cu_seqlens, block_size: int, stream=None):
    """Block keys [nblk_total, Hkv, 128] fp32."""
    lib = load()
    cu = _cu(cu_seqlens)
    nb = num_blocks(cu, block_size)
    kbar = torch.empty((nb, k.shape[1], k.shape[2]), dtype=torch.float32, device=k.device)
    dk, dc, db = map(describe, (k, cu, kbar))
    _check("moba_pool", lib.moba_pool(_ref(dk), _ref(dc), int(block_size), _ref(db),
                                      _stream(k, stream)))
    return kbar


def select(q, k, cu_seqlens, block_size: int, topk: int, nmax: int = 0, stream=None):
    """sel [T, Hq, topk] int32 (and scores [T, Hq, nmax] fp32 if nmax > 0)."""
    lib = load()
    cu = _cu(cu_seqlens)
    T, Hq = q.shape[0], q.shape[1]
    sel = torch.empty((T, Hq, topk), dtype=torch.int32, device=q.device)
    scores = torch.empty((T, Hq, nmax), dtype=torch.float32, device=q.device) if nmax > 0 else None
    dq, dk, dc, ds = map(describe, (q, k, cu, sel))
    dsc = describe(scores) if scores is not None else None
    _check("moba_select", lib.moba_select(_ref(dq), _ref(dk), _ref(dc), int(block_size), int(topk),
                                          _ref(ds), _ref(dsc), _stream(q, stream)))
    return (sel, scores) if nmax > 0 else sel


def route(sel, cu_seqlens, block_size: int, num_kv_heads: int, stream=None):
    """(counts [Hkv*nblk] int32, offsets [Hkv*nblk+1] int64, entries [E] int32)."""
    lib = load()
    cu = _cu(cu_seqlens)
    T, Hq, topk = sel.shape
    nb, E = route_size(cu, block_size, topk, Hq, stream)
    nbins = nb * num_kv_heads
    counts = torch.empty((nbins,), dtype=torch.int32, device=sel.device)
    offsets = torch.empty((nbins + 1,), dtype=torch.int64, device=sel.device)
    entries = torch.empty((E,), dtype=torch.int32, device=sel.device)
    ds, dc, dn, do, de = map(describe, (sel, cu, counts, offsets, entries))
    _check("moba_route", lib.moba_route(_ref(ds), _ref(dc), int(block_size), int(num_kv_heads),
                                        _ref(dn), _ref(do), _ref(de), _stream(sel, stream)))
    return counts, offsets, entries


def workspace_bytes(T: int, num_q_heads: int, num_kv_heads: int, nblk_total: int, topk: int,
                    head_dim: int = 128) -> int:
    """Device workspace bytes a one-pass moba_forward needs (an upper bound)."""
    return int(load().moba_workspace_bytes(int(T), int(num_q_heads), int(num_kv_heads),
                                           int(head_dim), int(nblk_total), int(topk)))


def workspace_held_bytes() -> int:
    """Bytes of device workspace the library holds on the current device."""
    return int(load().moba_workspace_held_bytes())


def take_wait_timeouts() -> int:
    """Give-ups of the backward's hand-over wait since the last call (waits
    for the device)."""
    n = ctypes.c_uint64()
    _check("moba_take_wait_timeouts", load().moba_take_wait_timeouts(ctypes.byref(n)))
    return int(n.value)


def release_workspace() -> None:
    _check("moba_release_workspace", load().moba_release_workspace())


def profile_enable(on: bool = True) -> None:
    load().moba_profile_enable(1 if on else 0)


def profile_read() -> dict:
    """{phase: (launches, total_ms)} since the last read."""
    buf = (PhaseStat * 32)()
    n = load().moba_profile_read(buf, 32)
    return {buf[i].name.decode(): (int(buf[i].launches), float(buf[i].total_ms)) for i in range(n)}

"""fp64 CPU oracle for MoBA's causal prefill forward pass (arXiv 2502.13189).

TEST INFRASTRUCTURE ONLY: the checker that the GPU library is compared against.
Only the tests, the smoke check and the benchmark's CPU-baseline leg import this
module; the product path never does.  It shares no code with the HIP library.

The arithmetic lives in ``moba_oracle.c`` (plain C, fp64, one loop nest per step
of the paper's definitions); this module only builds it with gcc and marshals
numpy arrays.  Inputs are numpy arrays shaped [T, H, D]: float32 for fp32 inputs
or uint16 holding bf16 bit patterns.  Row ids are r = t * Hq + h.

Functions and the passages they follow (Method section of the paper):
  pool    -- block mean of the keys (Eq. 6; Algorithm 1, mean_pool)
  select  -- unscaled gate scores, causal mask, forced current block, top-k
             (Eq. 5, Eq. 6; "Causality" and "Current Block Attention"
             paragraphs; the top-k footnote of the scaling-law experiments)
  attend  -- softmax over the selected blocks, causal inside the current block
             (Eq. 2, Eq. 4)
  dense   -- causal softmax attention (Eq. 1)
  forward -- pool, select, attend
  attend_backward -- gradients of attend w.r.t. q, k, v for a fixed selection
             (chain rule through Eq. 2; the hard gate of Eq. 3/5 passes none)
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moba_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libmoba_oracle.so")
_lib = None

_F32, _BF16 = 0, 1


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (portable x86-64 code, OpenMP over rows)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB_PATH)
        vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        lib.moba_oracle_pool.argtypes = [vp, i32, i64, i32, i32, vp, i32, i32, vp, vp]
        lib.moba_oracle_select.argtypes = [vp, i32, i64, i32, i32, i32, vp, i32, i32, i32, vp,
                                           vp, i64, vp, vp, i64, i32]
        lib.moba_oracle_attend.argtypes = [vp, vp, vp, i32, i64, i32, i32, i32, vp, i32, i32,
                                           i32, vp, vp, i64, vp, vp, i32]
        lib.moba_oracle_attend_backward.argtypes = [vp, vp, vp, vp, i32, i64, i32, i32, i32,
                                                    vp, i32, i32, i32, vp, vp, i64, i32, vp,
                                                    i64, i64, vp, vp, vp, vp, vp]
        lib.moba_oracle_dense.argtypes = [vp, vp, vp, i32, i64, i32, i32, i32, vp, i32, vp,
                                          i64, vp, vp]
        lib.moba_oracle_num_blocks.argtypes = [vp, i32, i32]
        lib.moba_oracle_threads.restype = ctypes.c_int
        lib.moba_oracle_set_threads.argtypes = [i32]
        _lib = lib
    return _lib


def threads() -> int:
    return _load().moba_oracle_threads()


def set_threads(n: int) -> None:
    _load().moba_oracle_set_threads(int(n))


def _elems(x: np.ndarray):
    x = np.ascontiguousarray(x)
    if x.dtype == np.float32:
        return x, _F32
    if x.dtype == np.uint16:
        return x, _BF16
    raise TypeError("oracle inputs must be float32 or uint16 (bf16 bits), got %s" % x.dtype)


def _cu(cu) -> np.ndarray:
    cu = np.ascontiguousarray(np.asarray(cu, dtype=np.int32))
    assert cu.ndim == 1 and cu.size >= 1
    return cu


def _rows(rows):
    if rows is None:
        return None, 0
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    return rows, rows.size


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(rc, what):
    if rc != 0:
        raise ValueError("oracle %s failed with code %d" % (what, rc))


def num_blocks(cu, block_size: int) -> int:
    cu = _cu(cu)
    return _load().moba_oracle_num_blocks(cu.ctypes.data, cu.size - 1, int(block_size))


def pool(k: np.ndarray, cu, block_size: int, with_abs: bool = False):
    """Block keys [nblk_total, Hkv, D] in fp64 (and mean |K| if with_abs)."""
    k, dt = _elems(k)
    T, Hkv, D = k.shape
    cu = _cu(cu)
    nb = num_blocks(cu, block_size)
    kbar = np.zeros((nb, Hkv, D), np.float64)
    kabs = np.zeros((nb, Hkv, D), np.float64) if with_abs else None
    _check(_load().moba_oracle_pool(k.ctypes.data, dt, T, Hkv, D, cu.ctypes.data, cu.size - 1,
                                    int(block_size), kbar.ctypes.data, _ptr(kabs)), "pool")
    return (kbar, kabs) if with_abs else kbar


def select(q: np.ndarray, kbar: np.ndarray, cu, block_size: int, topk: int, rows=None,
           nmax: int = 0):
    """sel [nrows, topk] int32 (ascending, -1 padded); with nmax > 0 also the
    unscaled scores [nrows, nmax] (NaN where j >= c)."""
    q, dt = _elems(q)
    T, Hq, D = q.shape
    Hkv = kbar.shape[1]
    cu = _cu(cu)
    rows, nr = _rows(rows)
    n = T * Hq if rows is None else nr
    sel = np.empty((n, topk), np.int32)
    sc = np.empty((n, nmax), np.float64) if nmax > 0 else None
    kbar = np.ascontiguousarray(kbar, dtype=np.float64)
    _check(_load().moba_oracle_select(q.ctypes.data, dt, T, Hq, Hkv, D, cu.ctypes.data,
                                      cu.size - 1, int(block_size), int(topk), kbar.ctypes.data,
                                      _ptr(rows), nr, sel.ctypes.data, _ptr(sc), int(nmax), 0),
           "select")
    return (sel, sc) if nmax > 0 else sel


def select_rows(q_rows: np.ndarray, T: int, Hq: int, kbar: np.ndarray, cu, block_size: int,
                topk: int, rows, nmax: int = 0):
    """select() for the listed rows given only their query vectors q_rows
    [nrows, D] (in the order of rows) of a [T, Hq, D] problem; with nmax > 0
    also the scores, as in select()."""
    q, dt = _elems(q_rows)
    D = q.shape[-1]
    Hkv = kbar.shape[1]
    cu = _cu(cu)
    rows, nr = _rows(rows)
    assert rows is not None and q.reshape(-1, D).shape[0] == nr
    sel = np.empty((nr, topk), np.int32)
    sc = np.empty((nr, nmax), np.float64) if nmax > 0 else None
    kbar = np.ascontiguousarray(kbar, dtype=np.float64)
    _check(_load().moba_oracle_select(q.ctypes.data, dt, int(T), int(Hq), Hkv, D, cu.ctypes.data,
                                      cu.size - 1, int(block_size), int(topk), kbar.ctypes.data,
                                      _ptr(rows), nr, sel.ctypes.data, _ptr(sc), int(nmax), 1),
           "select")
    return (sel, sc) if nmax > 0 else sel


def attend(q, k, v, cu, block_size: int, sel: np.ndarray, rows=None):
    """Attention over a given selection: out [nrows, D] fp64, lse [nrows] fp64."""
    q, dt = _elems(q)
    k, dtk = _elems(k)
    v, dtv = _elems(v)
    assert dt == dtk == dtv
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    cu = _cu(cu)
    rows, nr = _rows(rows)
    n = T * Hq if rows is None else nr
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    if sel.ndim != 2:
        sel = sel.reshape(n, -1)
    assert sel.shape[0] == n
    out = np.empty((n, D), np.float64)
    lse = np.empty((n,), np.float64)
    _check(_load().moba_oracle_attend(q.ctypes.data, k.ctypes.data, v.ctypes.data, dt, T, Hq,
                                      Hkv, D, cu.ctypes.data, cu.size - 1, int(block_size),
                                      sel.shape[1], sel.ctypes.data, _ptr(rows), nr,
                                      out.ctypes.data, lse.ctypes.data, 0), "attend")
    return out, lse


def attend_rows(q_rows, T: int, Hq: int, k, v, cu, block_size: int, sel: np.ndarray, rows):
    """attend() for the listed rows given only their query vectors q_rows
    [nrows, D] (in the order of rows) of a [T, Hq, D] problem."""
    q, dt = _elems(q_rows)
    k, dtk = _elems(k)
    v, dtv = _elems(v)
    assert dt == dtk == dtv
    D = q.shape[-1]
    Hkv = k.shape[1]
    cu = _cu(cu)
    rows, nr = _rows(rows)
    assert rows is not None and q.reshape(-1, D).shape[0] == nr
    sel = np.ascontiguousarray(sel, dtype=np.int32).reshape(nr, -1)
    out = np.empty((nr, D), np.float64)
    lse = np.empty((nr,), np.float64)
    _check(_load().moba_oracle_attend(q.ctypes.data, k.ctypes.data, v.ctypes.data, dt, int(T),
                                      int(Hq), Hkv, D, cu.ctypes.data, cu.size - 1,
                                      int(block_size), sel.shape[1], sel.ctypes.data, _ptr(rows),
                                      nr, out.ctypes.data, lse.ctypes.data, 1), "attend")
    return out, lse


def attend_backward(q, k, v, dout, cu, block_size: int, sel: np.ndarray, rows=None,
                    shape=None, want_dq: bool = True, kv_window=None, with_bounds: bool = False):
    """Gradients of attend() for a fixed selection sel [nrows, topk].

    Returns (dq, dk, dv): dq [nrows, D] fp64 (None unless want_dq); dk, dv
    [(hi - lo), Hkv, D] fp64 over the token window kv_window = (lo, hi)
    (None: no dk/dv; "all": every token), holding the listed rows'
    contributions.  With shape = (T, Hq), q and dout hold the listed rows'
    vectors only, [nrows, D] in list order.  With with_bounds, returns
    (dq, dk, dv, cq, ck, cv): the sums of absolute terms, in the same
    layouts, that the tests' rounding tolerances scale with."""
    q, dt = _elems(q)
    k, dtk = _elems(k)
    v, dtv = _elems(v)
    dout, dto = _elems(dout)
    assert dt == dtk == dtv == dto
    D = q.shape[-1]
    Hkv = k.shape[1]
    compact = shape is not None
    if compact:
        T, Hq = int(shape[0]), int(shape[1])
    else:
        T, Hq = q.shape[0], q.shape[1]
    cu = _cu(cu)
    rows, nr = _rows(rows)
    n = T * Hq if rows is None else nr
    if compact:
        assert rows is not None and q.reshape(-1, D).shape[0] == nr
        assert dout.reshape(-1, D).shape[0] == nr
    else:
        assert dout.shape == q.shape
    sel = np.ascontiguousarray(sel, dtype=np.int32).reshape(n, -1)
    dq = np.empty((n, D), np.float64) if want_dq else None
    lo, hi = 0, 0
    dk = dv = ck = cv = None
    if kv_window is not None:
        lo, hi = (0, T) if kv_window == "all" else (int(kv_window[0]), int(kv_window[1]))
        dk = np.empty((hi - lo, Hkv, D), np.float64)
        dv = np.empty((hi - lo, Hkv, D), np.float64)
        if with_bounds:
            ck = np.empty((hi - lo, Hkv, D), np.float64)
            cv = np.empty((hi - lo, Hkv, D), np.float64)
    cq = np.empty((n, D), np.float64) if (with_bounds and want_dq) else None
    _check(_load().moba_oracle_attend_backward(
        q.ctypes.data, k.ctypes.data, v.ctypes.data, dout.ctypes.data, dt, T, Hq, Hkv, D,
        cu.ctypes.data, cu.size - 1, int(block_size), sel.shape[1], sel.ctypes.data, _ptr(rows),
        nr, 1 if compact else 0, _ptr(dq), lo, hi, _ptr(dk), _ptr(dv), _ptr(cq), _ptr(ck),
        _ptr(cv)), "attend_backward")
    if with_bounds:
        return dq, dk, dv, cq, ck, cv
    return dq, dk, dv


def dense(q, k, v, cu, rows=None):
    """Dense causal attention: out [nrows, D] fp64, lse [nrows] fp64."""
    q, dt = _elems(q)
    k, dtk = _elems(k)
    v, dtv = _elems(v)
    assert dt == dtk == dtv
    T, Hq, D = q.shape
    Hkv = k.shape[1]
    cu = _cu(cu)
    rows, nr = _rows(rows)
    n = T * Hq if rows is None else nr
    out = np.empty((n, D), np.float64)
    lse = np.empty((n,), np.float64)
    _check(_load().moba_oracle_dense(q.ctypes.data, k.ctypes.data, v.ctypes.data, dt, T, Hq,
                                     Hkv, D, cu.ctypes.data, cu.size - 1, _ptr(rows), nr,
                                     out.ctypes.data, lse.ctypes.data), "dense")
    return out, lse


def forward(q, k, v, cu, block_size: int, topk: int, rows=None):
    """Full MoBA forward for the listed rows: (sel, out, lse)."""
    kbar = pool(k, cu, block_size)
    sel = select(q, kbar, cu, block_size, topk, rows=rows)
    out, lse = attend(q, k, v, cu, block_size, sel, rows=rows)
    return sel, out, lse

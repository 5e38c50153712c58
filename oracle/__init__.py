"""k-MIP attention CPU oracle (float64) -- TEST INFRASTRUCTURE ONLY.

The plain definition of k-MIP self-attention (Eq. 1 and Algorithm 1 of
arXiv 2604.03815) lives in ``kmip_oracle.c``; this module builds it with gcc
and wraps it with ctypes.  Only the test suite, ``__graft_entry__.smoke()``
and the benchmark's CPU-baseline leg may import it.  The GPU library never
links or calls it, and the two share no code.

Inputs are float64 arrays, node-major: Q and K [N, H, d_K], V and the output
gradient [N, H, d_V] (the value width may differ from the key width, Section
3.1).  ``from_bf16`` widens the
raw bfloat16 bits that the GPU path receives, exactly, so both sides see the
same values.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "kmip_oracle.c")
_LIB = os.path.join(_HERE, "libkmip_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (OpenMP over independent query rows)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", _SRC, "-o", tmp, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.oracle_topk.argtypes = [P, P, P, i32, i64, i32, i32, i32, i64, P, P, P, P]
        lib.oracle_attend.argtypes = [P, P, P, i64, i32, i32, i32, i32, f64, i64, P, P, P, f64, P, P]
        lib.oracle_forward.argtypes = [P, P, P, P, i32, i64, i32, i32, i32, i32, f64, P, P, P]
        lib.oracle_backward.argtypes = [P, P, P, P, i64, i32, i32, i32, i32, f64, P, P, f64, P, P, P]
        lib.oracle_check_set.argtypes = [P, P, P, i32, i64, i32, i32, i32, i64, P, P, P, P, P]
        lib.oracle_threads.argtypes = []
        for f in ("oracle_threads", "oracle_topk", "oracle_attend", "oracle_forward", "oracle_backward",
                  "oracle_check_set"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def from_bf16(b: np.ndarray) -> np.ndarray:
    """Exact float64 values of raw bfloat16 bits."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _f64(x):
    return np.ascontiguousarray(x, dtype=np.float64)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _shape(Q):
    if Q.ndim != 3:
        raise ValueError("expected [N, H, d]")
    return Q.shape


def _offsets(offsets, N):
    if offsets is None:
        return None, 1
    o = np.ascontiguousarray(offsets, dtype=np.int32)
    if o.ndim != 1 or len(o) < 2 or o[0] != 0 or o[-1] != N or np.any(np.diff(o) < 0):
        raise ValueError("graph offsets must start at 0, be non-decreasing and end at N")
    return o, len(o) - 1


def _sel(sel, N, H):
    if sel is None:
        return None, N * H
    s = np.ascontiguousarray(sel, dtype=np.int64)
    if s.size and (s.min() < 0 or s.max() >= N * H):
        raise ValueError("query-head id out of range")
    return s, s.size


def topk(Q, K, k: int, offsets=None, sel=None):
    """RowwiseTopK by full sort.  Returns (idx [nsel,k] int32, scores [nsel,k], next [nsel]).

    ``sel`` lists query-head ids i*H+h (default: all, in order).  ``next`` is
    the score of the (k+1)-th key (-inf when the graph has <= k nodes).
    """
    Q, K = _f64(Q), _f64(K)
    N, H, d = _shape(Q)
    o, G = _offsets(offsets, N)
    s, n = _sel(sel, N, H)
    idx = np.empty((n, k), np.int32)
    sc = np.empty((n, k), np.float64)
    nx = np.empty(n, np.float64)
    rc = _load().oracle_topk(_ptr(Q), _ptr(K), _ptr(o), G, N, H, d, k, n, _ptr(s),
                             _ptr(idx), _ptr(sc), _ptr(nx))
    if rc != 0:
        raise MemoryError("oracle_topk could not allocate")
    return idx, sc, nx


def _value_width(V, N, H, name="V"):
    if V.ndim != 3 or V.shape[0] != N or V.shape[1] != H:
        raise ValueError(f"{name} must be [N, H, d_V] with the N and H of Q")
    return V.shape[2]


def _key_shape(K, N, H, d):
    if K.shape != (N, H, d):
        raise ValueError("K must have the shape of Q")


def _keep(keep, n, k, drop_rate):
    """Dropout keep draws as uint8 [n, k] (or None) and the scale 1/(1 - rate)."""
    if not 0.0 <= drop_rate < 1.0:
        raise ValueError("drop_rate must lie in [0, 1)")
    if keep is None:
        if drop_rate != 0.0:
            raise ValueError("a drop rate needs keep draws")
        return None, 1.0
    keep = np.ascontiguousarray(keep, dtype=np.uint8).reshape(n, k)
    return keep, 1.0 / (1.0 - drop_rate)


def attend(Q, K, V, idx, scale: float, sel=None, keep=None, drop_rate: float = 0.0):
    """Softmax + aggregate on a given index set.  Returns (out [nsel,d_V], lse [nsel]).

    keep: optional dropout draws [nsel, k] (nonzero keeps a slot's weight,
    scaled by 1/(1 - drop_rate))."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    N, H, d = _shape(Q)
    _key_shape(K, N, H, d)
    dv = _value_width(V, N, H)
    s, n = _sel(sel, N, H)
    idx = np.ascontiguousarray(idx, dtype=np.int32).reshape(n, -1)
    k = idx.shape[1]
    kp, ks = _keep(keep, n, k, drop_rate)
    out = np.empty((n, dv), np.float64)
    lse = np.empty(n, np.float64)
    _load().oracle_attend(_ptr(Q), _ptr(K), _ptr(V), N, H, d, dv, k, float(scale), n, _ptr(s),
                          _ptr(idx), _ptr(kp), ks, _ptr(out), _ptr(lse))
    return out, lse


def forward(Q, K, V, k: int, scale: float, offsets=None):
    """Full forward.  Returns (out [N,H,d_V], idx [N,H,k], lse [N,H])."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    N, H, d = _shape(Q)
    _key_shape(K, N, H, d)
    dv = _value_width(V, N, H)
    o, G = _offsets(offsets, N)
    idx = np.empty((N, H, k), np.int32)
    out = np.empty((N, H, dv), np.float64)
    lse = np.empty((N, H), np.float64)
    rc = _load().oracle_forward(_ptr(Q), _ptr(K), _ptr(V), _ptr(o), G, N, H, d, dv, k,
                                float(scale), _ptr(idx), _ptr(out), _ptr(lse))
    if rc != 0:
        raise MemoryError("oracle_forward could not allocate")
    return out, idx, lse


def backward(Q, K, V, dO, idx, scale: float, keep=None, drop_rate: float = 0.0):
    """Gradients with the index set held fixed.  Returns (dQ [N,H,d_K], dK [N,H,d_K], dV [N,H,d_V]).

    keep, drop_rate: the forward's dropout draws [N, H, k] and rate."""
    Q, K, V, dO = _f64(Q), _f64(K), _f64(V), _f64(dO)
    N, H, d = _shape(Q)
    _key_shape(K, N, H, d)
    dv = _value_width(V, N, H)
    if dO.shape != V.shape:
        raise ValueError("dO must have the shape of V")
    idx = np.ascontiguousarray(idx, dtype=np.int32).reshape(N, H, -1)
    k = idx.shape[2]
    kp, ks = _keep(keep, N * H, k, drop_rate)
    dQ = np.empty((N, H, d), np.float64)
    dK = np.empty((N, H, d), np.float64)
    dV = np.empty((N, H, dv), np.float64)
    rc = _load().oracle_backward(_ptr(Q), _ptr(K), _ptr(V), _ptr(dO), N, H, d, dv, k,
                                 float(scale), _ptr(idx), _ptr(kp), ks, _ptr(dQ), _ptr(dK), _ptr(dV))
    if rc != 0:
        raise MemoryError("oracle_backward could not allocate")
    return dQ, dK, dV


def check_set(Q, K, idx, offsets=None, sel=None):
    """Exact-score check of a given index set.  Returns (min_in, max_out, flags)."""
    Q, K = _f64(Q), _f64(K)
    N, H, d = _shape(Q)
    o, G = _offsets(offsets, N)
    s, n = _sel(sel, N, H)
    idx = np.ascontiguousarray(idx, dtype=np.int32).reshape(n, -1)
    k = idx.shape[1]
    mn = np.empty(n, np.float64)
    mx = np.empty(n, np.float64)
    fl = np.empty(n, np.int32)
    _load().oracle_check_set(_ptr(Q), _ptr(K), _ptr(o), G, N, H, d, k, n, _ptr(s), _ptr(idx),
                             _ptr(mn), _ptr(mx), _ptr(fl))
    return mn, mx, fl


def threads() -> int:
    """OpenMP threads the oracle runs on."""
    return int(_load().oracle_threads())

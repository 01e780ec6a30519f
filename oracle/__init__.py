"""Float64 CPU oracle for exact dense softmax attention (ctypes wrapper).

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` are the only users.  The product path
(``paper_2112_05682_amd``) never imports this package, and this package never
imports the product.

The arithmetic lives in ``mea_oracle.c``; see its header for what each
function computes and which part of the paper it follows (Section 1 attention
definition, Section 3 running-max update, Section 4 chunk summaries and
combine, hand-derived backward).  This module only converts arrays to
contiguous float64 and calls the C entry points.

Layout of every tensor argument: ``[B, H, n, features]`` (feature index
innermost); q and k have d features, v, o and the upstream gradient d_v.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mea_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_i64 = ctypes.c_int64
_dbl = ctypes.c_double
_int = ctypes.c_int
_dp = ctypes.POINTER(ctypes.c_double)
_lp = ctypes.POINTER(ctypes.c_int64)


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra",
               "-Werror", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        full = [_i64, _i64, _i64, _i64, _i64, _i64, _dp, _dp, _dp, _dbl, _int, _lp]
        lib.mea_oracle_fwd.argtypes = full + [_dp, _dp]
        lib.mea_oracle_fwd_lazy.argtypes = full + [_dp, _dp]
        lib.mea_oracle_fwd_chunked.argtypes = full + [_i64, _i64, _dp, _dp]
        lib.mea_oracle_bwd.argtypes = [_i64] * 6 + [_dp] * 4 + [_dbl, _int, _lp] + [_dp] * 3
        head = [_i64, _i64, _i64, _i64, _dp, _dp, _dp]
        lib.mea_oracle_fwd_rows.argtypes = head + [_dbl, _int, _i64, _lp, _i64, _dp, _dp]
        lib.mea_oracle_bwd_dq_rows.argtypes = head + [_dp, _dbl, _int, _i64, _lp, _i64, _dp]
        lib.mea_oracle_bwd_dkdv_keys.argtypes = head + [_dp, _dbl, _int, _i64, _lp, _i64, _dp,
                                                        _dp]
        for name in ("mea_oracle_fwd", "mea_oracle_fwd_lazy", "mea_oracle_fwd_chunked",
                     "mea_oracle_bwd", "mea_oracle_fwd_rows", "mea_oracle_bwd_dq_rows",
                     "mea_oracle_bwd_dkdv_keys", "mea_oracle_num_threads"):
            getattr(lib, name).restype = _int
        lib.mea_oracle_num_threads.argtypes = []
        lib.mea_oracle_set_num_threads.argtypes = [_int]
        lib.mea_oracle_set_num_threads.restype = None
        _lib = lib
    return _lib


def _f64(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(_dp)


def _check(rc: int, name: str) -> None:
    if rc != 0:
        raise RuntimeError("%s failed with code %d" % (name, rc))


def _dims(q, k, v):
    """(B, H, n_q, n_k, d, d_v): q, k are [B, H, n, d], v is [B, H, n_k, d_v]."""
    if q.ndim != 4 or k.ndim != 4 or v.ndim != 4:
        raise ValueError("q, k, v must be [B, H, n, features]")
    B, H, nq, d = q.shape
    if k.shape[:2] != (B, H) or v.shape[:3] != k.shape[:3] or k.shape[3] != d:
        raise ValueError("shape mismatch: q %s k %s v %s" % (q.shape, k.shape, v.shape))
    return B, H, nq, k.shape[2], d, v.shape[3]


def _kv_len(kv_len, batch: int):
    """Per-batch valid key lengths as a contiguous int64 array (None: all keys)."""
    if kv_len is None:
        return None
    a = np.ascontiguousarray(np.asarray(kv_len, dtype=np.int64).reshape(-1))
    if a.size != batch:
        raise ValueError("kv_len must have one entry per batch")
    return a


def _lptr(a):
    return a.ctypes.data_as(_lp) if a is not None else None


def default_scale(d: int) -> float:
    """The 1/sqrt(d) query scaling of the paper's implementation (Section 4)."""
    return 1.0 / float(np.sqrt(d))


def num_threads() -> int:
    return int(_load().mea_oracle_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads of the oracle's later calls from this thread."""
    _load().mea_oracle_set_num_threads(int(n))


def fwd(q, k, v, scale=None, causal=False, kv_len=None):
    """Direct form.  Returns (o [B,H,n_q,d], lse [B,H,n_q]) in float64.
    ``kv_len``: optional per-batch valid key lengths (key padding)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, nq, nk, d, dv = _dims(q, k, v)
    scale = default_scale(d) if scale is None else float(scale)
    kl = _kv_len(kv_len, B)
    o = np.empty((B, H, nq, dv))
    lse = np.empty((B, H, nq))
    _check(_load().mea_oracle_fwd(B, H, nq, nk, d, dv, _ptr(q), _ptr(k), _ptr(v), scale,
                                  int(bool(causal)), _lptr(kl), _ptr(o), _ptr(lse)),
           "mea_oracle_fwd")
    return o, lse


def fwd_lazy(q, k, v, scale=None, causal=False, kv_len=None):
    """Section 3 single-pass form.  Returns (o, lse)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, nq, nk, d, dv = _dims(q, k, v)
    scale = default_scale(d) if scale is None else float(scale)
    kl = _kv_len(kv_len, B)
    o = np.empty((B, H, nq, dv))
    lse = np.empty((B, H, nq))
    _check(_load().mea_oracle_fwd_lazy(B, H, nq, nk, d, dv, _ptr(q), _ptr(k), _ptr(v), scale,
                                       int(bool(causal)), _lptr(kl), _ptr(o), _ptr(lse)),
           "mea_oracle_fwd_lazy")
    return o, lse


def fwd_chunked(q, k, v, scale=None, causal=False, query_chunk=1024, key_chunk=4096,
                kv_len=None):
    """Section 4 chunk-summary form.  Returns (o, lse)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    B, H, nq, nk, d, dv = _dims(q, k, v)
    scale = default_scale(d) if scale is None else float(scale)
    kl = _kv_len(kv_len, B)
    o = np.empty((B, H, nq, dv))
    lse = np.empty((B, H, nq))
    _check(_load().mea_oracle_fwd_chunked(B, H, nq, nk, d, dv, _ptr(q), _ptr(k), _ptr(v), scale,
                                          int(bool(causal)), _lptr(kl), int(query_chunk),
                                          int(key_chunk), _ptr(o), _ptr(lse)),
           "mea_oracle_fwd_chunked")
    return o, lse


def bwd(q, k, v, dout, scale=None, causal=False, kv_len=None):
    """Hand-derived gradients.  Returns (dq, dk, dv) in float64."""
    q, k, v, dout = _f64(q), _f64(k), _f64(v), _f64(dout)
    B, H, nq, nk, d, d_v = _dims(q, k, v)
    if dout.shape != (B, H, nq, d_v):
        raise ValueError("dout must be [B, H, n_q, d_v]")
    scale = default_scale(d) if scale is None else float(scale)
    kl = _kv_len(kv_len, B)
    dq = np.empty_like(q)
    dk = np.empty_like(k)
    dv = np.empty_like(v)
    _check(_load().mea_oracle_bwd(B, H, nq, nk, d, d_v, _ptr(q), _ptr(k), _ptr(v), _ptr(dout),
                                  scale, int(bool(causal)), _lptr(kl), _ptr(dq), _ptr(dk),
                                  _ptr(dv)),
           "mea_oracle_bwd")
    return dq, dk, dv


def _head(x):
    x = _f64(x)
    if x.ndim != 2:
        raise ValueError("expected one head [n, d]")
    return x


def _n_valid(n_valid, n_k: int) -> int:
    return n_k if n_valid is None else int(n_valid)


def fwd_rows(q, k, v, rows, scale=None, causal=False, n_valid=None):
    """Forward for selected query rows of one head (q, k, v are [n, d]);
    ``n_valid``: keys visible at most (key padding), default all."""
    q, k, v = _head(q), _head(k), _head(v)
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    d, dv = q.shape[1], v.shape[1]
    scale = default_scale(d) if scale is None else float(scale)
    o = np.empty((rows.size, dv))
    lse = np.empty(rows.size)
    _check(_load().mea_oracle_fwd_rows(q.shape[0], k.shape[0], d, dv, _ptr(q), _ptr(k), _ptr(v),
                                       scale, int(bool(causal)), _n_valid(n_valid, k.shape[0]),
                                       rows.ctypes.data_as(_lp), rows.size, _ptr(o), _ptr(lse)),
           "mea_oracle_fwd_rows")
    return o, lse


def bwd_dq_rows(q, k, v, dout, rows, scale=None, causal=False, n_valid=None):
    """dQ for selected query rows of one head."""
    q, k, v, dout = _head(q), _head(k), _head(v), _head(dout)
    rows = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    d, dv = q.shape[1], v.shape[1]
    scale = default_scale(d) if scale is None else float(scale)
    dq = np.empty((rows.size, d))
    _check(_load().mea_oracle_bwd_dq_rows(q.shape[0], k.shape[0], d, dv, _ptr(q), _ptr(k), _ptr(v),
                                          _ptr(dout), scale, int(bool(causal)),
                                          _n_valid(n_valid, k.shape[0]),
                                          rows.ctypes.data_as(_lp), rows.size, _ptr(dq)),
           "mea_oracle_bwd_dq_rows")
    return dq


def bwd_dkdv_keys(q, k, v, dout, keys, scale=None, causal=False, n_valid=None):
    """dK and dV for selected key rows of one head."""
    q, k, v, dout = _head(q), _head(k), _head(v), _head(dout)
    keys = np.ascontiguousarray(np.asarray(keys, dtype=np.int64))
    d, d_v = q.shape[1], v.shape[1]
    scale = default_scale(d) if scale is None else float(scale)
    dk = np.empty((keys.size, d))
    dv = np.empty((keys.size, d_v))
    _check(_load().mea_oracle_bwd_dkdv_keys(q.shape[0], k.shape[0], d, d_v, _ptr(q), _ptr(k),
                                            _ptr(v), _ptr(dout), scale, int(bool(causal)),
                                            _n_valid(n_valid, k.shape[0]),
                                            keys.ctypes.data_as(_lp), keys.size, _ptr(dk),
                                            _ptr(dv)),
           "mea_oracle_bwd_dkdv_keys")
    return dk, dv

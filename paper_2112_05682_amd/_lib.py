"""ctypes loader for ``libmea.so`` (the HIP library built from ``csrc/``).

Only argument marshalling lives here.  The library is loaded from this package
directory; if it is missing the call fails loudly -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmea.so")

MEA_OK = 0
MEA_ERR_INVALID_ARG = 1
MEA_ERR_UNSUPPORTED = 2
MEA_ERR_WORKSPACE = 3
MEA_ERR_HIP = 4
MEA_ERR_SCRATCH = 5

# Static scratch of mea_attention_bwd_noalloc (MEA_NOALLOC_SCRATCH_BYTES).
NOALLOC_SCRATCH_BYTES = (16 << 20) + 256

MEA_F32, MEA_F16, MEA_BF16 = 0, 1, 2

# Every entry point declared in include/mea.h.
EXPORTS = (
    "mea_attention_fwd_workspace_size",
    "mea_attention_bwd_workspace_size",
    "mea_attention_fwd",
    "mea_attention_bwd",
    "mea_attention_bwd_noalloc",
    "mea_status_string",
)


class MeaTensorStrides(ctypes.Structure):
    """Mirror of ``mea_tensor_strides`` (elements)."""

    _fields_ = [("batch", ctypes.c_int64), ("head", ctypes.c_int64), ("row", ctypes.c_int64)]


class MeaStrides(ctypes.Structure):
    """Mirror of ``mea_strides``."""

    _fields_ = [(name, MeaTensorStrides) for name in ("q", "k", "v", "o", "d_o", "dq", "dk", "dv")]


class MeaProblem(ctypes.Structure):
    """Mirror of ``mea_problem``."""

    _fields_ = [
        ("batch", ctypes.c_int64),
        ("heads", ctypes.c_int64),
        ("n_q", ctypes.c_int64),
        ("n_k", ctypes.c_int64),
        ("d", ctypes.c_int64),
        ("dtype", ctypes.c_int32),
        ("causal", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("out_f32", ctypes.c_int32),
        ("strides", ctypes.POINTER(MeaStrides)),
        ("kv_len", ctypes.c_void_p),
        ("d_v", ctypes.c_int64),
    ]


class MeaError(RuntimeError):
    def __init__(self, name: str, status: int, message: str):
        super().__init__("%s failed: %s (status %d)" % (name, message, status))
        self.status = status


_lib = None


def load(path: str = LIB_PATH):
    """Load the library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(
            "libmea.so not found at %s: build it with `python -m paper_2112_05682_amd.build` "
            "(the attention path has no fallback)" % path)
    lib = ctypes.CDLL(path)
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    prob = ctypes.POINTER(MeaProblem)
    lib.mea_attention_fwd_workspace_size.argtypes = [prob, ctypes.POINTER(sz)]
    lib.mea_attention_bwd_workspace_size.argtypes = [prob, ctypes.POINTER(sz)]
    lib.mea_attention_fwd.argtypes = [prob, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.mea_attention_bwd.argtypes = [prob, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.mea_attention_bwd_noalloc.argtypes = [prob, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    for name in ("mea_attention_fwd_workspace_size", "mea_attention_bwd_workspace_size",
                 "mea_attention_fwd", "mea_attention_bwd", "mea_attention_bwd_noalloc"):
        getattr(lib, name).restype = ctypes.c_int
    lib.mea_status_string.argtypes = [ctypes.c_int]
    lib.mea_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load().mea_status_string(int(status)).decode()


def check(name: str, status: int) -> None:
    if status != MEA_OK:
        raise MeaError(name, status, status_string(status))


def problem(batch, heads, n_q, n_k, d, dtype, causal, scale, out_f32=False,
            strides: dict | None = None, kv_len: int | None = None,
            d_v: int | None = None) -> MeaProblem:
    """``strides`` maps tensor names (q, k, v, o, d_o, dq, dk, dv) to
    (batch, head, row) element strides; missing names and None mean contiguous
    [B, H, n, width].  ``kv_len`` is the device address of an int32 [B] array of
    valid key lengths (key padding), or None.  ``d_v``: head dimension of v, o,
    do and dv (None: d)."""
    dv = int(d) if d_v is None else int(d_v)
    p = MeaProblem(int(batch), int(heads), int(n_q), int(n_k), int(d), int(dtype),
                   int(bool(causal)), float(scale), int(bool(out_f32)), None,
                   int(kv_len) if kv_len else None, 0 if dv == int(d) else dv)
    if strides:
        st = MeaStrides()
        for name, n, w in (("q", n_q, d), ("k", n_k, d), ("v", n_k, dv), ("o", n_q, dv),
                           ("d_o", n_q, dv), ("dq", n_q, d), ("dk", n_k, d), ("dv", n_k, dv)):
            bs, hs, rs = strides.get(name) or (int(heads) * int(n) * int(w), int(n) * int(w), int(w))
            setattr(st, name, MeaTensorStrides(int(bs), int(hs), int(rs)))
        p._strides_keepalive = st  # the struct must outlive the calls that read it
        p.strides = ctypes.pointer(st)
    return p


def fwd_workspace_size(p: MeaProblem) -> int:
    out = ctypes.c_size_t(0)
    check("mea_attention_fwd_workspace_size",
          load().mea_attention_fwd_workspace_size(ctypes.byref(p), ctypes.byref(out)))
    return int(out.value)


def bwd_workspace_size(p: MeaProblem) -> int:
    out = ctypes.c_size_t(0)
    check("mea_attention_bwd_workspace_size",
          load().mea_attention_bwd_workspace_size(ctypes.byref(p), ctypes.byref(out)))
    return int(out.value)


def fwd(p: MeaProblem, q, k, v, o, lse, o_lo, workspace, workspace_bytes, stream) -> int:
    """Raw call; pointers are ints (device addresses) or None, returns the status."""
    return load().mea_attention_fwd(ctypes.byref(p), q, k, v, o, lse, o_lo, workspace,
                                    workspace_bytes, stream)


def bwd(p: MeaProblem, q, k, v, o, o_lo, d_o, lse, dq, dk, dv, workspace, workspace_bytes,
        stream) -> int:
    return load().mea_attention_bwd(ctypes.byref(p), q, k, v, o, o_lo, d_o, lse, dq, dk, dv,
                                    workspace, workspace_bytes, stream)


def bwd_noalloc(p: MeaProblem, q, k, v, o, o_lo, d_o, lse, dq, dk, dv, stream) -> int:
    """The backward without a workspace argument (static device scratch)."""
    return load().mea_attention_bwd_noalloc(ctypes.byref(p), q, k, v, o, o_lo, d_o, lse, dq, dk,
                                            dv, stream)

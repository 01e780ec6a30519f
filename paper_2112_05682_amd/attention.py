"""PyTorch-facing wrapper of the C ABI: allocation of outputs and workspace
through torch, and the current HIP stream.  Every step of the computation runs
in the HIP kernels of ``libmea.so``; nothing here computes attention.

Tensors are ``[B, H, n, d]`` on one GPU with contiguous features; their batch,
head and row strides are passed to the kernels, so views such as the paper's
``[n, heads, d]`` layout (a transpose of ``[B, n, H, d]``) or slices of a
packed QKV projection are read and written in place.  q, k, v and the
gradients share one dtype (float32, float16 or bfloat16), o and do share it or
are float32 (16-bit inputs with a float32 output, as in the paper's
experiments); d must be 64 or 128.
"""
from __future__ import annotations

import math

import torch

from . import _lib

_DTYPE_CODE = {torch.float32: _lib.MEA_F32, torch.float16: _lib.MEA_F16,
               torch.bfloat16: _lib.MEA_BF16}


def _problem(q: torch.Tensor, k: torch.Tensor, causal: bool, scale, out_f32: bool = False,
             tensors: dict | None = None, kv_len: torch.Tensor | None = None):
    """``tensors`` maps ABI tensor names (q, k, v, o, d_o, dq, dk, dv) to the
    tensors of a call, whose strides are passed when any is not contiguous.
    ``kv_len``: int32 [B] tensor on q's device (valid keys per batch) or None."""
    if q.dim() != 4 or k.dim() != 4:
        raise ValueError("q and k must be [B, H, n, d]")
    B, H, n_q, d = q.shape
    n_k = k.shape[2]
    d_v = tensors["v"].shape[3] if tensors and tensors.get("v") is not None else d
    if q.dtype not in _DTYPE_CODE:
        raise TypeError("unsupported dtype %s" % q.dtype)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    strides = None
    if tensors and any(not t.is_contiguous() for t in tensors.values() if t is not None):
        strides = {name: tuple(t.stride()[:3]) for name, t in tensors.items() if t is not None}
    if kv_len is not None:
        if kv_len.dtype != torch.int32 or kv_len.device != q.device or tuple(kv_len.shape) != (B,) \
                or not kv_len.is_contiguous():
            raise ValueError("kv_len must be a contiguous int32 [B] tensor on q's device")
    return _lib.problem(B, H, n_q, n_k, d, _DTYPE_CODE[q.dtype], causal, scale,
                        out_f32 and q.dtype != torch.float32, strides,
                        kv_len.data_ptr() if kv_len is not None else None, d_v)


def _check_tensors(names, tensors, dtype, device):
    for name, t in zip(names, tensors):
        if not t.is_cuda:
            raise ValueError("%s must be a GPU tensor" % name)
        if t.device != device:
            raise ValueError("%s is on %s, expected %s" % (name, t.device, device))
        if t.dtype != dtype:
            raise TypeError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
        if name == "lse":
            if not t.is_contiguous():
                raise ValueError("lse must be contiguous")
            continue
        if t.dim() != 4 or t.stride(3) != 1:
            raise ValueError("%s must be [B, H, n, d] with contiguous features" % name)
        unit = 16 // t.element_size()
        if t.data_ptr() % 16 or any(st_ % unit for st_ in t.stride()[:3]):
            raise ValueError("%s: data pointer and strides must be multiples of 16 bytes" % name)


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def fwd_workspace_bytes(q, k, causal=False, scale=None) -> int:
    return _lib.fwd_workspace_size(_problem(q, k, causal, scale))


def bwd_workspace_bytes(q, k, causal=False, scale=None) -> int:
    return _lib.bwd_workspace_size(_problem(q, k, causal, scale))


def attention_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, causal: bool = False,
                  scale: float | None = None, need_lse: bool = True, out=None,
                  out_dtype: torch.dtype | None = None, kv_len: torch.Tensor | None = None,
                  residual: bool = False):
    """Returns ``(o, lse)``; ``lse`` is float32 ``[B, H, n_q]`` (None if not needed).
    ``out_dtype`` is q's dtype (default) or torch.float32.  ``kv_len`` (int32
    ``[B]`` on the GPU) masks keys ``j >= kv_len[b]`` of batch b (key padding);
    a row with no visible key gets o = 0 and lse = -inf.  With ``residual``
    the call returns ``(o, lse, o_lo)``: for a 16-bit o, ``o_lo`` is o's
    rounding residual (contiguous, o's dtype), which the backward uses to form
    D_i = do_i . o_i accurately where the softmax saturates; None for a
    float32 o."""
    if k.shape[:3] != v.shape[:3] or q.shape[:2] != k.shape[:2] or q.shape[3] != k.shape[3]:
        raise ValueError("shape mismatch: q %s k %s v %s" % (tuple(q.shape), tuple(k.shape),
                                                              tuple(v.shape)))
    o_shape = tuple(q.shape[:3]) + (v.shape[3],)  # o has v's head dimension
    _check_tensors(("q", "k", "v"), (q, k, v), q.dtype, q.device)
    out_dtype = q.dtype if out_dtype is None else out_dtype
    if out_dtype not in (q.dtype, torch.float32):
        raise TypeError("out_dtype must be q's dtype or float32")
    o = torch.empty(o_shape, dtype=out_dtype, device=q.device) if out is None else out
    _check_tensors(("out",), (o,), out_dtype, q.device)
    if tuple(o.shape) != o_shape:
        raise ValueError("out must be [B, H, n_q, d_v]")
    p = _problem(q, k, causal, scale, out_dtype == torch.float32,
                 {"q": q, "k": k, "v": v, "o": o}, kv_len)
    lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device) if need_lse else None
    o_lo = torch.empty(o_shape, dtype=out_dtype, device=q.device) \
        if residual and out_dtype != torch.float32 else None
    ws_bytes = _lib.fwd_workspace_size(p)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device) if ws_bytes else None
    _lib.check("mea_attention_fwd", _lib.fwd(
        p, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
        lse.data_ptr() if lse is not None else None,
        o_lo.data_ptr() if o_lo is not None else None,
        ws.data_ptr() if ws is not None else None, ws_bytes, _stream(q.device)))
    return (o, lse, o_lo) if residual else (o, lse)


def attention_bwd(q, k, v, o, lse, do, causal: bool = False, scale: float | None = None,
                  need_dq: bool = True, need_dkdv: bool = True, out=None,
                  kv_len: torch.Tensor | None = None, o_lo: torch.Tensor | None = None):
    """Returns ``(dq, dk, dv)`` for the upstream gradient ``do``; a gradient that
    is not needed is returned as None and its kernel is not run.  ``out`` may
    give the (dq, dk, dv) tensors to write (any may be None: allocated).
    ``kv_len`` must be the forward's; masked keys get zero dk and dv rows.
    ``o_lo``: the forward's residual of a 16-bit o (``attention_fwd(...,
    residual=True)``); without it D_i is formed from the rounded o alone."""
    _check_tensors(("q", "k", "v"), (q, k, v), q.dtype, q.device)
    if o.dtype not in (q.dtype, torch.float32):
        raise TypeError("o must have q's dtype or float32")
    _check_tensors(("o", "do"), (o, do), o.dtype, q.device)
    _check_tensors(("lse",), (lse,), torch.float32, q.device)
    o_shape = tuple(q.shape[:3]) + (v.shape[3],)
    if tuple(o.shape) != o_shape or tuple(do.shape) != o_shape or tuple(lse.shape) != tuple(q.shape[:3]):
        raise ValueError("o, do must be [B, H, n_q, d_v] and lse [B, H, n_q]")
    if o_lo is not None:
        _check_tensors(("o_lo",), (o_lo,), o.dtype, q.device)
        if tuple(o_lo.shape) != o_shape or not o_lo.is_contiguous():
            raise ValueError("o_lo must be a contiguous [B, H, n_q, d_v] tensor")
    if not (need_dq or need_dkdv):
        raise ValueError("nothing to compute")
    given = out if out is not None else (None, None, None)
    dq = (given[0] if given[0] is not None else torch.empty(q.shape, dtype=q.dtype, device=q.device)) \
        if need_dq else None
    dk = (given[1] if given[1] is not None else torch.empty(k.shape, dtype=k.dtype, device=k.device)) \
        if need_dkdv else None
    dv = (given[2] if given[2] is not None else torch.empty(v.shape, dtype=v.dtype, device=v.device)) \
        if need_dkdv else None
    outs = [(n_, t) for n_, t in (("dq", dq), ("dk", dk), ("dv", dv)) if t is not None]
    _check_tensors([n_ for n_, _ in outs], [t for _, t in outs], q.dtype, q.device)
    for n_, t in outs:
        if t.shape != {"dq": q.shape, "dk": k.shape, "dv": v.shape}[n_]:
            raise ValueError("%s has the wrong shape" % n_)
    p = _problem(q, k, causal, scale, o.dtype == torch.float32,
                 {"q": q, "k": k, "v": v, "o": o, "d_o": do, "dq": dq, "dk": dk, "dv": dv}, kv_len)
    ws_bytes = _lib.bwd_workspace_size(p)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
    _lib.check("mea_attention_bwd", _lib.bwd(
        p, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
        o_lo.data_ptr() if o_lo is not None else None, do.data_ptr(),
        lse.data_ptr(), dq.data_ptr() if need_dq else None,
        dk.data_ptr() if need_dkdv else None, dv.data_ptr() if need_dkdv else None,
        ws.data_ptr(), ws_bytes,
        _stream(q.device)))
    return dq, dk, dv


class MemoryEfficientAttention(torch.autograd.Function):
    """Autograd wrapper: saves q, k, v, o, the O(n) lse and, for a 16-bit o,
    o's rounding residual (O(n d), like o)."""

    @staticmethod
    def forward(ctx, q, k, v, causal=False, scale=None, out_dtype=None, kv_len=None):
        q, k, v = (_feature_contiguous(t) for t in (q, k, v))
        o, lse, o_lo = attention_fwd(q, k, v, causal, scale, need_lse=True, out_dtype=out_dtype,
                                     kv_len=kv_len, residual=True)
        ctx.save_for_backward(q, k, v, o, lse, o_lo)
        ctx.causal = causal
        ctx.scale = scale
        ctx.kv_len = kv_len
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse, o_lo = ctx.saved_tensors
        dq, dk, dv = attention_bwd(q, k, v, o, lse, _feature_contiguous(do.to(o.dtype)), ctx.causal,
                                   ctx.scale, kv_len=ctx.kv_len, o_lo=o_lo)
        return dq, dk, dv, None, None, None, None


def _feature_contiguous(t: torch.Tensor) -> torch.Tensor:
    """t itself when the kernels can read it in place (contiguous features,
    16-byte aligned pointer and strides), else a contiguous copy."""
    unit = 16 // t.element_size()
    if t.dim() == 4 and t.stride(3) == 1 and t.data_ptr() % 16 == 0 and \
            all(st_ % unit == 0 for st_ in t.stride()[:3]):
        return t
    return t.contiguous()


class PackedQKVAttention(torch.autograd.Function):
    """Self-attention on the output of one fused QKV projection, ``qkv`` of
    shape ``[B, n, 3, H, d]``: q, k and v are read as strided views of it, the
    output is ``[B, n, H, d]`` (so ``reshape(B, n, H * d)`` is free) and the
    gradient is written as one packed ``[B, n, 3, H, d]`` tensor -- neither
    direction copies or transposes.  Saves qkv, o, the O(n) lse and o's
    rounding residual."""

    @staticmethod
    def forward(ctx, qkv, causal=False, scale=None, kv_len=None):
        if qkv.dim() != 5 or qkv.shape[2] != 3:
            raise ValueError("qkv must be [B, n, 3, H, d]")
        qkv = qkv if qkv.is_contiguous() else qkv.contiguous()
        B, n, _, H, d = qkv.shape
        q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))  # [B, H, n, d] views
        o = torch.empty(B, n, H, d, dtype=qkv.dtype, device=qkv.device)
        _, lse, o_lo = attention_fwd(q, k, v, causal, scale, need_lse=True, out=o.transpose(1, 2),
                                     kv_len=kv_len, residual=True)
        ctx.save_for_backward(qkv, o, lse, o_lo)
        ctx.causal, ctx.scale, ctx.kv_len = causal, scale, kv_len
        return o

    @staticmethod
    def backward(ctx, do):
        qkv, o, lse, o_lo = ctx.saved_tensors
        q, k, v = (qkv[:, :, i].transpose(1, 2) for i in range(3))
        dqkv = torch.empty_like(qkv)
        dq, dk, dv = (dqkv[:, :, i].transpose(1, 2) for i in range(3))
        do_ = _feature_contiguous(do.to(o.dtype).transpose(1, 2))
        attention_bwd(q, k, v, o.transpose(1, 2), lse, do_, ctx.causal, ctx.scale, out=(dq, dk, dv),
                      kv_len=ctx.kv_len, o_lo=o_lo)
        return dqkv, None, None, None


def attention_packed(qkv, causal: bool = False, scale: float | None = None,
                     kv_len: torch.Tensor | None = None):
    """Exact softmax self-attention of a packed ``[B, n, 3, H, d]`` projection,
    differentiable, O(n) extra memory; returns ``[B, n, H, d]``.  ``kv_len``:
    optional int32 ``[B]`` valid key lengths (key padding)."""
    return PackedQKVAttention.apply(qkv, causal, scale, kv_len)


def attention(q, k, v, causal: bool = False, scale: float | None = None,
              out_dtype: torch.dtype | None = None, kv_len: torch.Tensor | None = None):
    """Exact softmax attention, differentiable, O(n) extra memory.  ``kv_len``:
    optional int32 ``[B]`` valid key lengths (keys ``j >= kv_len[b]`` masked)."""
    return MemoryEfficientAttention.apply(q, k, v, causal, scale, out_dtype, kv_len)

"""The allocation-free backward entry point, mea_attention_bwd_noalloc.

Its per-row workspace lives in a static device array instead of a caller
buffer; the kernels are mea_attention_bwd's.  The GPU test calls both entry
points through the C ABI on the same inputs and requires identical results,
twice in a row with the second problem smaller than the first (the array
keeps the first call's contents).  The CPU tests check the rejections that
happen before any HIP call.
"""
import ctypes

import pytest
import torch

from paper_2112_05682_amd import _lib, attention_bwd, attention_fwd
from paper_2112_05682_amd.attention import _problem
from paper_2112_05682_amd.inputs import attention_inputs

FAKE = 0x10000  # aligned non-null address; only used where validation must fail first


def test_noalloc_is_declared_and_exported():
    lib = _lib.load()
    assert ctypes.cast(lib.mea_attention_bwd_noalloc, ctypes.c_void_p).value
    assert "static scratch" in _lib.status_string(_lib.MEA_ERR_SCRATCH)


@pytest.mark.parametrize("d,rows_limit", [(64, 1 << 20), (128, 1 << 21)])
def test_noalloc_rejects_problems_beyond_the_scratch(d, rows_limit):
    # B * H * ceil(n_q / 64) * 64 padded rows: at the limit the workspace fits
    # exactly; 64 rows more are rejected before anything is enqueued (the
    # pointers are fake, so reaching a launch would fault -- it must not).
    heads = rows_limit // 16384
    at = _lib.problem(1, heads, 16384, 128, d, _lib.MEA_BF16, False, d ** -0.5)
    assert _lib.bwd_workspace_size(at) <= _lib.NOALLOC_SCRATCH_BYTES
    over = _lib.problem(1, heads, 16384 + 1, 128, d, _lib.MEA_BF16, False, d ** -0.5)
    assert _lib.bwd_workspace_size(over) > _lib.NOALLOC_SCRATCH_BYTES
    assert _lib.bwd_noalloc(over, *([FAKE] * 10), None) == _lib.MEA_ERR_SCRATCH


def test_noalloc_validates_like_the_backward():
    p = _lib.problem(1, 2, 100, 100, 64, _lib.MEA_BF16, False, 0.125)
    ptrs = [FAKE] * 10
    ptrs[0] = None  # q
    assert _lib.bwd_noalloc(p, *ptrs, None) == _lib.MEA_ERR_INVALID_ARG
    ptrs = [FAKE] * 10
    ptrs[7], ptrs[8], ptrs[9] = None, None, None  # nothing requested
    assert _lib.bwd_noalloc(p, *ptrs, None) == _lib.MEA_ERR_INVALID_ARG
    bad = _lib.problem(1, 2, 100, 100, 96, _lib.MEA_BF16, False, 0.125)
    assert _lib.bwd_noalloc(bad, *([FAKE] * 10), None) == _lib.MEA_ERR_UNSUPPORTED


def _both(B, H, nq, nk, d, dtype, causal):
    print("noalloc case B=%d H=%d nq=%d nk=%d d=%d %s causal=%s" % (B, H, nq, nk, d, dtype, causal),
          flush=True)
    x = {k_: t.to("cuda") for k_, t in attention_inputs(B, H, nq, nk, d, dtype).items()}
    q, k, v, do = x["q"], x["k"], x["v"], x["do"]
    o, lse, o_lo = attention_fwd(q, k, v, causal=causal, residual=True)
    ref = attention_bwd(q, k, v, o, lse, do, causal=causal, o_lo=o_lo)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    p = _problem(q, k, causal, None, False, {"q": q, "k": k, "v": v, "o": o, "d_o": do,
                                             "dq": dq, "dk": dk, "dv": dv})
    assert _lib.bwd_workspace_size(p) <= _lib.NOALLOC_SCRATCH_BYTES
    st = _lib.bwd_noalloc(p, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                          o_lo.data_ptr() if o_lo is not None else None, do.data_ptr(),
                          lse.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                          torch.cuda.current_stream().cuda_stream)
    _lib.check("mea_attention_bwd_noalloc", st)
    torch.cuda.synchronize()
    for name, a, b in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
        assert torch.equal(a, b), name


@pytest.mark.gpu
@pytest.mark.parametrize("d,dtype", [(64, "bf16"), (128, "bf16"), (64, "fp32")])
def test_noalloc_matches_the_backward_on_two_calls(d, dtype):
    # 16-bit d = 64 runs the two-group kernels (records in the scratch), the
    # others the float32 per-row arrays; the second call is smaller.
    _both(2, 4, 1000, 1200, d, dtype, True)
    _both(1, 2, 300, 257, d, dtype, False)

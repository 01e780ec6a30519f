"""GPU parity of the backward pass against the float64 oracle's hand-derived
gradients.  The GPU backward consumes the GPU forward's O, LSE and (for a 16-bit
O) O's rounding residual, as the autograd path does in training; the oracle
recomputes everything from Q, K, V, dO.  Each gradient is held to the bar per
tensor and per row (see parity_util)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2112_05682_amd import attention, attention_bwd, attention_fwd
from paper_2112_05682_amd.inputs import WORKLOADS, attention_inputs, workload_inputs
from parity_util import TOL, check, f64, gradient_row_scales, to_gpu

pytestmark = pytest.mark.gpu


def gpu_grads(g, causal, out_dtype=None, residual=True):
    """Forward then backward through the C ABI; with `residual` (the default,
    as in training) a 16-bit o's rounding residual goes from one to the other."""
    o, lse, o_lo = attention_fwd(g["q"], g["k"], g["v"], causal=causal, out_dtype=out_dtype,
                                 residual=True)
    dq, dk, dv = attention_bwd(g["q"], g["k"], g["v"], o, lse, g["do"].to(o.dtype),
                               causal=causal, o_lo=o_lo if residual else None)
    torch.cuda.synchronize()
    return dq, dk, dv


def run_and_compare(B, H, nq, nk, d, dtype, causal, std=1.0, qk_mult=1.0, out_dtype=None,
                    residual=True, row_tol=None):
    print("case B=%d H=%d nq=%d nk=%d d=%d %s causal=%s mult=%s out=%s residual=%s" % (
        B, H, nq, nk, d, dtype, causal, qk_mult, out_dtype, residual), flush=True)
    x = attention_inputs(B, H, nq, nk, d, dtype, std, qk_mult)
    dq, dk, dv = gpu_grads(to_gpu(x), causal, out_dtype, residual)
    # dO is drawn in the input dtype, so its float32 copy is exact for the oracle too.
    args = (f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["do"]))
    rq, rk, rv = oracle.bwd(*args, scale=d ** -0.5, causal=causal)
    _, rl = oracle.fwd(*args[:3], scale=d ** -0.5, causal=causal)
    cq, ck = gradient_row_scales(*args, rl, d ** -0.5, causal)
    for name, got, ref, terms in (("dQ", dq, rq, cq), ("dK", dk, rk, ck), ("dV", dv, rv, None)):
        check(name, f64(got), ref, TOL[dtype], row_tol, terms=terms)


SHAPES = [(1, 1, 1, 1), (1, 2, 7, 100), (2, 3, 129, 257), (1, 1, 700, 700), (1, 2, 300, 70),
          (1, 1, 64, 1500)]


@pytest.mark.parametrize("dtype", ["fp32", "bf16", "fp16"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_backward_small(dtype, d, causal, shape):
    run_and_compare(*shape, d, dtype, causal)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("shape", [(1, 2, 7, 100), (2, 1, 300, 257), (1, 1, 64, 1500)],
                         ids=lambda s: "x".join(map(str, s)))
def test_backward_float32_output(dtype, d, causal, shape):
    # 16-bit inputs with a float32 o / do (the paper's experimental setting).
    run_and_compare(*shape, d, dtype, causal, out_dtype=torch.float32)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_backward_large_logits(dtype, d, causal):
    # Q, K scaled by 30 (logits ~1e3, Section 3's stability setting).  The
    # softmax saturates, so the true dS_ij = w_ij (dO_i . v_j - D_i) is a tiny
    # difference and D_i = dO_i . O_i must be accurate: o in the input dtype
    # (the default) with the forward's rounding residual.
    run_and_compare(1, 2, 300, 500, d, dtype, causal, qk_mult=30.0)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_backward_large_logits_float32_output(d, causal):
    # The paper's setting (16-bit inputs, float32 o): no residual exists.
    run_and_compare(1, 2, 300, 500, d, "bf16", causal, qk_mult=30.0, out_dtype=torch.float32)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_backward_without_residual_ordinary_inputs(d, causal):
    # Without the residual (o_lo = NULL) D comes from the rounded o alone:
    # within the bar for inputs whose softmax does not saturate.
    run_and_compare(2, 2, 300, 257, d, "bf16", causal, residual=False)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("nq", [2048, 2049])
def test_backward_causal_d64_both_kernels(dtype, nq):
    # Causal 16-bit d = 64 problems of up to 2048 queries run the 4-wave
    # backward (per-row values as two arrays), longer ones the two-group
    # kernels (records): both sides of the switch.
    run_and_compare(1, 1, nq, nq, 64, dtype, True)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("shape", [(2, 3, 512, 700), (2, 3, 513, 700), (1, 2, 100, 40000)],
                         ids=lambda s: "x".join(map(str, s)))
def test_backward_unmasked_d64_both_kernels(dtype, shape):
    # Unmasked 16-bit d = 64 problems of up to 512 queries run the 4-wave
    # backward, longer ones the two-group kernels: both sides of the switch,
    # and few queries against many keys.
    B, H, nq, nk = shape
    run_and_compare(B, H, nq, nk, 64, dtype, False)


def test_backward_fp32_self_attention_n256():
    w = WORKLOADS["selfattn_fp32_b1h1_n256_d64"]
    run_and_compare(w.batch, w.heads, w.n_q, w.n_k, w.d, w.dtype, w.causal)


def sampled(n, count, seed):
    rng = np.random.default_rng(seed)
    idx = rng.choice(n, size=count - 2, replace=False)
    return np.unique(np.concatenate([[0, n - 1], idx]))


@pytest.mark.parametrize("name", ["selfattn_bf16_b1h16_n16384_d64",
                                  "causal_bf16_b4h32_n8192_d128"])
def test_backward_full_size_sampled(name):
    # Full-size workloads: the oracle recomputes sampled dQ rows and sampled
    # dK / dV rows of a few (batch, head) slices.
    w = WORKLOADS[name]
    print("workload", name, flush=True)
    x = workload_inputs(w)
    dq, dk, dv = gpu_grads(to_gpu(x), w.causal)
    dq, dk, dv = dq.cpu(), dk.cpu(), dv.cpu()
    for b, h in sorted({(0, 0), (w.batch - 1, w.heads - 1)}):
        args = (f64(x["q"][b, h]), f64(x["k"][b, h]), f64(x["v"][b, h]), f64(x["do"][b, h]))
        rows = sampled(w.n_q, 32, 7 + h)
        keys = sampled(w.n_k, 32, 9 + h)
        rq = oracle.bwd_dq_rows(*args, rows, scale=w.d ** -0.5, causal=w.causal)
        rk, rv = oracle.bwd_dkdv_keys(*args, keys, scale=w.d ** -0.5, causal=w.causal)
        print("  slice", (b, h), flush=True)
        check("dQ", f64(dq[b, h, rows]), rq, TOL[w.dtype])
        check("dK", f64(dk[b, h, keys]), rk, TOL[w.dtype])
        check("dV", f64(dv[b, h, keys]), rv, TOL[w.dtype])
    for t in (dq, dk, dv):
        assert torch.isfinite(t).all()


def test_backward_is_deterministic():
    g = to_gpu(attention_inputs(1, 3, 900, 1100, 64, "bf16"))
    a = gpu_grads(g, True)
    b = gpu_grads(g, True)
    for x, y in zip(a, b):
        assert torch.equal(x, y)


def test_autograd_function_matches_direct_calls():
    g = to_gpu(attention_inputs(2, 2, 200, 300, 64, "bf16"))
    q = g["q"].clone().requires_grad_()
    k = g["k"].clone().requires_grad_()
    v = g["v"].clone().requires_grad_()
    o = attention(q, k, v, causal=True)
    o.backward(g["do"])
    dq, dk, dv = gpu_grads(g, True)
    assert torch.equal(q.grad, dq) and torch.equal(k.grad, dk) and torch.equal(v.grad, dv)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("causal", [False, True])
def test_float32_output_backward_matches_the_staging_path(dtype, d, causal):
    # With float32 o and dO, mea_attention_bwd rounds dO to the input dtype in
    # the preprocess and runs the kernels of 16-bit outputs on the copy; the
    # allocation-free entry point keeps no copy and runs the kernels that
    # round dO while staging it.  The rounding is the same, so the gradients
    # must be bitwise equal (and within the bar against the oracle, which the
    # float32-output cases above check).
    from paper_2112_05682_amd import _lib
    from paper_2112_05682_amd.attention import _problem
    B, H, nq, nk = 2, 3, 700, 650
    print("f32-out staging case", dtype, d, causal, flush=True)
    x = to_gpu(attention_inputs(B, H, nq, nk, d, dtype))
    q, k, v = x["q"], x["k"], x["v"]
    o, lse = attention_fwd(q, k, v, causal=causal, out_dtype=torch.float32)
    do = x["do"].to(torch.float32)
    ref = attention_bwd(q, k, v, o, lse, do, causal=causal)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    p = _problem(q, k, causal, None, True, {"q": q, "k": k, "v": v, "o": o, "d_o": do,
                                            "dq": dq, "dk": dk, "dv": dv})
    st = _lib.bwd_noalloc(p, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), None, do.data_ptr(),
                          lse.data_ptr(), dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                          torch.cuda.current_stream().cuda_stream)
    _lib.check("mea_attention_bwd_noalloc", st)
    torch.cuda.synchronize()
    for name, a, b in zip(("dq", "dk", "dv"), (dq, dk, dv), ref):
        assert torch.equal(a, b), name

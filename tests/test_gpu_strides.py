"""GPU parity of strided tensors: the kernels read and write [B, H, n, d]
tensors through batch, head and row strides (features contiguous).

* The paper's [n, heads, d] layout: tensors stored as [B, n, H, d] and passed
  as transposed views, forward and backward, for the query-tiled, two-group,
  decode and key-split paths.
* Gradients written into strided views of caller-provided buffers.
* A packed QKV projection [B, n, 3, H, d] read in place and its gradient
  written packed (``attention_packed``).
* One key head shared by all query heads (head stride 0 for k and v).
Every case is compared with the float64 oracle on the same (widened) values.
"""
import pytest
import torch

import oracle
from paper_2112_05682_amd import attention_bwd, attention_fwd, attention_packed
from paper_2112_05682_amd.inputs import attention_inputs
from parity_util import TOL, TORCH_DT, check, check_lse, f64, gradient_row_scales

pytestmark = pytest.mark.gpu


def as_bnhd_view(t: torch.Tensor) -> torch.Tensor:
    """A [B, H, n, d] CPU tensor stored on the GPU as [B, n, H, d], returned as
    the [B, H, n, d] view of that storage (not contiguous)."""
    return t.transpose(1, 2).contiguous().to("cuda").transpose(1, 2)


CASES = [  # B, H, nq, nk, d, dtype, causal
    (2, 3, 300, 257, 64, "bf16", False),     # two-group kernels
    (1, 2, 200, 1000, 64, "fp16", True),
    (2, 2, 129, 300, 128, "bf16", False),    # 4-wave kernels
    (1, 3, 150, 200, 64, "fp32", True),
    (2, 4, 5, 3000, 64, "bf16", False),      # decode kernel
    (1, 2, 40, 2000, 128, "fp16", False),
    (1, 2, 256, 40000, 64, "bf16", False),   # key splits + staged combine
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_paper_layout_forward_and_backward(case):
    B, H, nq, nk, d, dtype, causal = case
    print("strided case", case, flush=True)
    x = attention_inputs(B, H, nq, nk, d, dtype, with_grad=True)
    g = {k: as_bnhd_view(t) for k, t in x.items()}
    assert not g["q"].is_contiguous()
    o, lse, o_lo = attention_fwd(g["q"], g["k"], g["v"], causal=causal, residual=True)
    # Gradients into strided views of [B, n, H, d] buffers.
    bufs = {n_: torch.empty(B, t.shape[2], H, d, dtype=TORCH_DT[dtype], device="cuda")
            for n_, t in (("dq", x["q"]), ("dk", x["k"]), ("dv", x["v"]))}
    views = tuple(bufs[n_].transpose(1, 2) for n_ in ("dq", "dk", "dv"))
    attention_bwd(g["q"], g["k"], g["v"], o, lse, g["do"], causal=causal, out=views, o_lo=o_lo)
    torch.cuda.synchronize()
    qq, kk, vv, dd = (f64(x[n_]) for n_ in ("q", "k", "v", "do"))
    ro, rl = oracle.fwd(qq, kk, vv, causal=causal)
    rdq, rdk, rdv = oracle.bwd(qq, kk, vv, dd, causal=causal)
    cq, ck = gradient_row_scales(qq, kk, vv, dd, rl, d ** -0.5, causal)
    for name, got, ref, t_ in (("O", o, ro, None), ("dQ", views[0], rdq, cq), ("dK", views[1], rdk, ck),
                               ("dV", views[2], rdv, None)):
        check(name, f64(got), ref, TOL[dtype], terms=t_)
    check_lse(f64(lse), rl)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("nq", [48, 333])
def test_packed_qkv_forward_and_backward(dtype, d, nq):
    B, H = 2, 2
    print("packed case", dtype, d, nq, flush=True)
    gen = torch.Generator().manual_seed(11)
    qkv = torch.randn(B, nq, 3, H, d, generator=gen).to(TORCH_DT[dtype])
    up = torch.randn(B, nq, H, d, generator=gen).to(TORCH_DT[dtype])
    t = qkv.to("cuda").requires_grad_(True)
    o = attention_packed(t, causal=True)
    o.backward(up.to("cuda"))
    torch.cuda.synchronize()
    assert o.shape == (B, nq, H, d) and t.grad.shape == qkv.shape
    q, k, v = (f64(qkv[:, :, i].transpose(1, 2)) for i in range(3))
    ro, rl = oracle.fwd(q, k, v, causal=True)
    rdq, rdk, rdv = oracle.bwd(q, k, v, f64(up.transpose(1, 2)), causal=True)
    cq, ck = gradient_row_scales(q, k, v, f64(up.transpose(1, 2)), rl, d ** -0.5, True)
    grad = t.grad.cpu()
    for name, got, ref, t_ in (("O", o.transpose(1, 2), ro, None),
                               ("dQ", grad[:, :, 0].transpose(1, 2), rdq, cq),
                               ("dK", grad[:, :, 1].transpose(1, 2), rdk, ck),
                               ("dV", grad[:, :, 2].transpose(1, 2), rdv, None)):
        check(name, f64(got), ref, TOL[dtype], terms=t_)


@pytest.mark.parametrize("nq", [1, 200])
def test_one_key_head_shared_by_all_query_heads(nq):
    # k and v of one head, read by H query heads through head stride 0.
    B, H, nk, d = 2, 4, 1500, 64
    x = attention_inputs(B, 1, nq, nk, d, "bf16", with_grad=False)
    q = attention_inputs(B, H, nq, nk, d, "bf16", seeds=(7, 8, 9, 10), with_grad=False)["q"]
    k = x["k"].to("cuda").expand(B, H, nk, d)
    v = x["v"].to("cuda").expand(B, H, nk, d)
    assert k.stride(1) == 0
    o, lse = attention_fwd(q.to("cuda"), k, v)
    torch.cuda.synchronize()
    ro, rl = oracle.fwd(f64(q), f64(x["k"].expand(B, H, nk, d)), f64(x["v"].expand(B, H, nk, d)))
    check("O", f64(o), ro, TOL["bf16"])
    check_lse(f64(lse), rl)

"""The drop-in layers of ``paper_2112_05682_amd.nn`` on the GPU.

* The multi-head attention module (projections in torch, attention in the HIP
  kernels) against the same module evaluated in float64 on the CPU with the
  oracle's attention and hand-derived attention gradients (Section 5.2):
  output, input gradient and weight gradients.
* A small causal Transformer language model on synthetic tokens trains
  through the kernels (mixed precision, one fixed batch): the loss is finite
  and falls, and the step time is printed (the paper trains a Transformer with
  this attention, Section 5; its data and comparison systems are not here).
"""
import time

import numpy as np
import pytest
import torch

import oracle
from paper_2112_05682_amd.nn import MultiheadAttention, TransformerLM
from parity_util import f64, rel_err

pytestmark = pytest.mark.gpu


class OracleAttention(torch.autograd.Function):
    """float64 CPU attention from the oracle, differentiable through its
    hand-derived backward."""

    @staticmethod
    def forward(ctx, q, k, v, causal, kv_len=None):
        o, _ = oracle.fwd(q.numpy(), k.numpy(), v.numpy(), causal=causal, kv_len=kv_len)
        ctx.save_for_backward(q, k, v)
        ctx.causal, ctx.kv_len = causal, kv_len
        return torch.from_numpy(o)

    @staticmethod
    def backward(ctx, do):
        q, k, v = ctx.saved_tensors
        dq, dk, dv = oracle.bwd(q.numpy(), k.numpy(), v.numpy(), do.contiguous().numpy(),
                                causal=ctx.causal, kv_len=ctx.kv_len)
        return torch.from_numpy(dq), torch.from_numpy(dk), torch.from_numpy(dv), None, None


def reference_mha(m: MultiheadAttention, x: torch.Tensor, kv_len=None) -> torch.Tensor:
    """The module's computation in float64 on the CPU with the oracle's attention."""
    B, n, E = x.shape
    H, d = m.num_heads, m.head_dim
    qkv = torch.nn.functional.linear(x, m.qkv.weight, m.qkv.bias)
    qkv = qkv.view(B, n, 3, H, d).permute(2, 0, 3, 1, 4)
    q, k, v = (t.contiguous() for t in qkv.unbind(0))
    o = OracleAttention.apply(q, k, v, m.causal, kv_len)
    return torch.nn.functional.linear(o.transpose(1, 2).reshape(B, n, E), m.out.weight, m.out.bias)


TOLS = {torch.float32: 1e-4, torch.bfloat16: 3e-2}


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16], ids=["fp32", "bf16"])
@pytest.mark.parametrize("d,kv_len", [(64, None), (128, None), (64, [50, 77])],
                         ids=["d64", "d128", "d64-padded"])
@pytest.mark.parametrize("causal", [False, True])
def test_mha_module_matches_oracle_composition(dtype, d, kv_len, causal):
    print("mha case", dtype, d, kv_len, causal, flush=True)
    torch.manual_seed(0)
    B, n, H = 2, 77, 2
    E = H * d
    m = MultiheadAttention(E, H, causal=causal, device="cuda", dtype=dtype)
    x = torch.randn(B, n, E, generator=torch.Generator().manual_seed(1)).to("cuda", dtype)
    g = torch.randn(B, n, E, generator=torch.Generator().manual_seed(2)).to("cuda", dtype)
    x.requires_grad_(True)
    kl = torch.tensor(kv_len, dtype=torch.int32, device="cuda") if kv_len else None
    y = m(x, kl)
    y.backward(g)
    torch.cuda.synchronize()

    # The same weights and inputs, widened exactly to float64.
    mr = MultiheadAttention.__new__(MultiheadAttention)
    torch.nn.Module.__init__(mr)
    mr.embed_dim, mr.num_heads, mr.head_dim, mr.causal = E, H, d, causal
    mr.qkv = torch.nn.Linear(E, 3 * E, dtype=torch.float64)
    mr.out = torch.nn.Linear(E, E, dtype=torch.float64)
    with torch.no_grad():
        for dst, src in ((mr.qkv, m.qkv), (mr.out, m.out)):
            dst.weight.copy_(src.weight.detach().to("cpu", torch.float64))
            dst.bias.copy_(src.bias.detach().to("cpu", torch.float64))
    xr = x.detach().to("cpu", torch.float64).requires_grad_(True)
    yr = reference_mha(mr, xr, kv_len)
    yr.backward(g.to("cpu", torch.float64))

    tol = TOLS[dtype]
    pairs = {"y": (y, yr), "dx": (x.grad, xr.grad), "dW_qkv": (m.qkv.weight.grad, mr.qkv.weight.grad),
             "db_qkv": (m.qkv.bias.grad, mr.qkv.bias.grad), "dW_out": (m.out.weight.grad, mr.out.weight.grad)}
    for name, (a, b) in pairs.items():
        e = rel_err(f64(a), b.detach().numpy())
        print("  %s rel_err %.3g" % (name, e), flush=True)
        assert np.isfinite(e) and e <= tol, (name, e)


def test_transformer_lm_trains_on_synthetic_tokens():
    torch.manual_seed(0)
    vocab, E, H, depth, n, B = 1024, 512, 8, 2, 1024, 4
    model = TransformerLM(vocab, E, H, depth, max_len=n, device="cuda")
    opt = torch.optim.AdamW(model.parameters(), lr=3e-4)
    gen = torch.Generator().manual_seed(5)
    tokens = torch.randint(0, vocab, (B, n + 1), generator=gen).to("cuda")
    inp, tgt = tokens[:, :-1], tokens[:, 1:]
    losses, times = [], []
    for step in range(30):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        with torch.autocast("cuda", dtype=torch.bfloat16):
            logits = model(inp)
        loss = torch.nn.functional.cross_entropy(logits.float().reshape(-1, vocab), tgt.reshape(-1))
        opt.zero_grad(set_to_none=True)
        loss.backward()
        opt.step()
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
        losses.append(float(loss.detach()))
    print("loss first %.3f last %.3f; step %.2f ms (median of the last 20), %.0f tokens/s" % (
        losses[0], losses[-1], 1e3 * float(np.median(times[10:])), B * n / float(np.median(times[10:]))),
        flush=True)
    assert all(np.isfinite(losses))
    # One fixed batch: the model memorises it, so the loss must fall well
    # below the uniform-guess level ln(vocab) it starts near.
    assert 0.8 * np.log(vocab) < losses[0] < 1.2 * np.log(vocab)
    assert losses[-1] < losses[0] - 1.0
    for p_ in model.parameters():
        assert p_.grad is not None and torch.isfinite(p_.grad).all()

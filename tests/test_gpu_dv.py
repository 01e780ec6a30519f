"""GPU parity with a value head dimension d_v different from the query/key
one (d, d_v in {64, 128}): q and k have d features, v, o, dO and dV have d_v.

These problems run the 4-wave kernels (the two-group and decode kernels need
d = d_v), including the key-split path with its staged combine, causal and
key-padded cases and a float32 output; every case against the float64 oracle
with the same widths.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2112_05682_amd import attention, attention_bwd, attention_fwd
from paper_2112_05682_amd.inputs import attention_inputs
from parity_util import TOL, check, check_lse, f64, gradient_row_scales, to_gpu

pytestmark = pytest.mark.gpu

CASES = [  # B, H, nq, nk, d, d_v, dtype, causal, kv_len, out_f32
    (2, 2, 300, 257, 64, 128, "bf16", False, None, False),
    (2, 2, 300, 300, 128, 64, "bf16", True, None, False),
    (1, 3, 150, 200, 64, 128, "fp16", True, [180], False),
    (2, 2, 129, 300, 128, 64, "fp32", False, None, False),
    (2, 2, 130, 200, 64, 128, "fp32", True, None, False),
    (2, 2, 40, 2000, 64, 128, "bf16", False, None, False),      # few queries (no decode kernel)
    (1, 1, 256, 40000, 128, 64, "bf16", False, None, False),    # key splits + staged combine
    (2, 2, 300, 257, 64, 128, "bf16", False, [200, 0], True),   # padding, float32 output
]


def _ids(c):
    return "x".join(map(str, c[:8])) + ("-kv" + "_".join(map(str, c[8])) if c[8] else "") + \
        ("-f32o" if c[9] else "")


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_value_width_matches_oracle(case):
    B, H, nq, nk, d, d_v, dtype, causal, kv_len, out_f32 = case
    print("d_v case", _ids(case), flush=True)
    x = attention_inputs(B, H, nq, nk, d, dtype, with_grad=True, d_v=d_v)
    g = to_gpu(x)
    kl = torch.tensor(kv_len, dtype=torch.int32, device="cuda") if kv_len else None
    o, lse, o_lo = attention_fwd(g["q"], g["k"], g["v"], causal=causal, kv_len=kl,
                                 out_dtype=torch.float32 if out_f32 else None, residual=True)
    assert tuple(o.shape) == (B, H, nq, d_v)
    do = g["do"].to(o.dtype)
    dq, dk, dv = attention_bwd(g["q"], g["k"], g["v"], o, lse, do, causal=causal, kv_len=kl,
                               o_lo=o_lo)
    torch.cuda.synchronize()
    qq, kk, vv = (f64(x[n_]) for n_ in ("q", "k", "v"))
    dd = f64(do)
    ro, rl = oracle.fwd(qq, kk, vv, causal=causal, kv_len=kv_len)
    rdq, rdk, rdv = oracle.bwd(qq, kk, vv, dd, causal=causal, kv_len=kv_len)
    cq, ck = gradient_row_scales(qq, kk, vv, dd, rl, d ** -0.5, causal, kv_len)
    terms = {"dQ": cq, "dK": ck}
    got = {"O": f64(o), "LSE": f64(lse), "dQ": f64(dq), "dK": f64(dk), "dV": f64(dv)}
    ref = {"O": ro, "LSE": rl, "dQ": rdq, "dK": rdk, "dV": rdv}
    tol = TOL[dtype]
    for b in range(B):
        n = nk if kv_len is None else max(0, min(kv_len[b], nk))
        if n == 0:
            assert np.all(got["O"][b] == 0.0) and np.all(got["LSE"][b] == -np.inf)
            assert all(np.all(got[k_][b] == 0.0) for k_ in ("dQ", "dK", "dV"))
            continue
        print("  batch", b, flush=True)
        for name in ("O", "dQ", "dK", "dV"):
            check(name, got[name][b], ref[name][b], tol, lead=1,
                  terms=terms[name][b] if name in terms else None)
        check_lse(got["LSE"][b], ref["LSE"][b])


def test_value_width_autograd():
    B, H, nq, nk, d, d_v = 2, 2, 130, 150, 128, 64
    x = attention_inputs(B, H, nq, nk, d, "bf16", with_grad=True, d_v=d_v)
    g = to_gpu(x)
    q, k, v = (g[n_].clone().requires_grad_(True) for n_ in ("q", "k", "v"))
    o = attention(q, k, v, causal=True)
    o.backward(g["do"])
    torch.cuda.synchronize()
    qq, kk, vv, dd = (f64(x[n_]) for n_ in ("q", "k", "v", "do"))
    ro, _ = oracle.fwd(qq, kk, vv, causal=True)
    rdq, rdk, rdv = oracle.bwd(qq, kk, vv, dd, causal=True)
    for name, got, ref in (("o", o, ro), ("dq", q.grad, rdq), ("dk", k.grad, rdk), ("dv", v.grad, rdv)):
        check(name, f64(got), ref, TOL["bf16"])

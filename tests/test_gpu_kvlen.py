"""GPU parity of key padding (``kv_len``): batch b sees only keys
j < kv_len[b] (clamped to [0, n_k]), on top of the causal mask.

Every kernel family is covered -- the two-group kernels (16-bit, d = 64), the
4-wave kernels (d = 128, float32), the decode kernel (n_q <= 64) and the
key-split path with its staged combine -- against the float64 oracle with the
same lengths.  A batch with no visible key must give o = 0, lse = -inf and
zero gradients exactly; padded keys must get dk = dv = 0 exactly; the values
stored at padded positions must not change any output (bitwise); and
kv_len = n_k must reproduce the unpadded call bitwise.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2112_05682_amd import attention, attention_bwd, attention_fwd
from paper_2112_05682_amd.inputs import attention_inputs
from parity_util import TOL, check, check_lse, f64, gradient_row_scales, to_gpu

pytestmark = pytest.mark.gpu

CASES = [  # B, H, nq, nk, d, dtype, causal, kv_len, out_f32
    (3, 2, 300, 257, 64, "bf16", False, [257, 100, 1], False),   # two-group kernels
    (3, 2, 300, 300, 64, "bf16", True, [300, 64, 0], False),
    (2, 2, 200, 1000, 64, "fp16", True, [999, 130], False),
    (2, 2, 300, 257, 64, "bf16", False, [200, 0], True),         # float32 output
    (3, 2, 129, 300, 128, "bf16", False, [300, 65, 0], False),   # 4-wave kernels
    (2, 2, 129, 300, 128, "fp16", True, [17, 280], False),
    (2, 3, 150, 200, 64, "fp32", True, [200, 33], False),
    (3, 4, 5, 3000, 64, "bf16", False, [3000, 1234, 0], False),  # decode kernel
    (2, 2, 40, 2000, 128, "fp16", True, [1, 1999], False),
    (2, 2, 48, 3000, 128, "bf16", False, [3000, 1001], False),   # two sub-tiles, swizzled rows
    (2, 1, 256, 40000, 64, "bf16", False, [40000, 777], False),  # key splits + staged combine
    (2, 2, 100, 300, 64, "bf16", False, [-5, 1 << 20], False),   # lengths clamp to [0, n_k]
]


def _ids(c):
    return "x".join(map(str, c[:7])) + "-kv" + "_".join(map(str, c[7])) + ("-f32o" if c[8] else "")


def _run(x, causal, kv_len, out_f32):
    g = to_gpu(x)
    kl = torch.tensor(kv_len, dtype=torch.int32, device="cuda") if kv_len is not None else None
    o, lse, o_lo = attention_fwd(g["q"], g["k"], g["v"], causal=causal, kv_len=kl,
                                 out_dtype=torch.float32 if out_f32 else None, residual=True)
    do = g["do"].to(o.dtype)
    dq, dk, dv = attention_bwd(g["q"], g["k"], g["v"], o, lse, do, causal=causal, kv_len=kl,
                               o_lo=o_lo)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_key_padding_matches_oracle(case):
    B, H, nq, nk, d, dtype, causal, kv_len, out_f32 = case
    print("kv_len case", _ids(case), flush=True)
    x = attention_inputs(B, H, nq, nk, d, dtype, with_grad=True)
    o, lse, dq, dk, dv = _run(x, causal, kv_len, out_f32)
    qq, kk, vv = (f64(x[n_]) for n_ in ("q", "k", "v"))
    # The oracle's upstream gradient is the one the kernels read (rounded to o's dtype).
    dd = f64(x["do"].to(o.dtype))
    ro, rl = oracle.fwd(qq, kk, vv, causal=causal, kv_len=kv_len)
    rdq, rdk, rdv = oracle.bwd(qq, kk, vv, dd, causal=causal, kv_len=kv_len)
    go, gl, gdq, gdk, gdv = (f64(t) for t in (o, lse, dq, dk, dv))
    cq, ck = gradient_row_scales(qq, kk, vv, dd, rl, d ** -0.5, causal, kv_len)
    tol = TOL[dtype]
    for b, n in enumerate(kv_len):
        n = max(0, min(n, nk))
        if n == 0:  # no visible key: exact zeros and -inf
            assert np.all(go[b] == 0.0) and np.all(gl[b] == -np.inf)
            assert np.all(gdq[b] == 0.0) and np.all(gdk[b] == 0.0) and np.all(gdv[b] == 0.0)
            continue
        assert np.all(gdk[b, :, n:] == 0.0) and np.all(gdv[b, :, n:] == 0.0), "padded keys"
        print("  batch", b, "valid keys", n, flush=True)
        for name, got_, ref_, t_ in (("O", go, ro, None), ("dQ", gdq, rdq, cq), ("dK", gdk, rdk, ck),
                                     ("dV", gdv, rdv, None)):
            check(name, got_[b], ref_[b], tol, lead=1, terms=t_[b] if t_ is not None else None)
        check_lse(gl[b], rl[b])


@pytest.mark.parametrize("case", [CASES[0], CASES[4], CASES[7], CASES[10]], ids=_ids)
def test_padded_values_do_not_matter_and_full_length_is_unpadded(case):
    B, H, nq, nk, d, dtype, causal, kv_len, out_f32 = case
    print("kv_len invariance", _ids(case), flush=True)
    x = attention_inputs(B, H, nq, nk, d, dtype, with_grad=True)
    base = _run(x, causal, kv_len, out_f32)
    y = dict(x)
    y["k"], y["v"] = x["k"].clone(), x["v"].clone()
    for b, n in enumerate(kv_len):
        n = max(0, min(n, nk))
        y["k"][b, :, n:] = 1000.0  # large logits at padded positions must not leak
        y["v"][b, :, n:] = -1000.0
    other = _run(y, causal, kv_len, out_f32)
    for name, a, b_ in zip(("o", "lse", "dq", "dk", "dv"), base, other):
        assert torch.equal(a, b_), name
    full = _run(x, causal, [nk] * B, out_f32)
    none = _run(x, causal, None, out_f32)
    for name, a, b_ in zip(("o", "lse", "dq", "dk", "dv"), full, none):
        assert torch.equal(a, b_), name


def test_autograd_with_key_padding():
    B, H, nq, nk, d = 2, 2, 130, 200, 64
    x = attention_inputs(B, H, nq, nk, d, "bf16", with_grad=True)
    kv_len = [150, 7]
    g = to_gpu(x)
    q, k, v = (g[n_].clone().requires_grad_(True) for n_ in ("q", "k", "v"))
    o = attention(q, k, v, causal=False, kv_len=torch.tensor(kv_len, dtype=torch.int32,
                                                             device="cuda"))
    o.backward(g["do"])
    torch.cuda.synchronize()
    qq, kk, vv, dd = (f64(x[n_]) for n_ in ("q", "k", "v", "do"))
    ro, _ = oracle.fwd(qq, kk, vv, kv_len=kv_len)
    rdq, rdk, rdv = oracle.bwd(qq, kk, vv, dd, kv_len=kv_len)
    for name, got, ref in (("o", o, ro), ("dq", q.grad, rdq), ("dk", k.grad, rdk),
                           ("dv", v.grad, rdv)):
        check(name, f64(got), ref, TOL["bf16"])

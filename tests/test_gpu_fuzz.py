"""Seeded random sweep of small problems through every kernel family, forward
and backward, against the float64 oracle.

Each case draws batch and head counts, query and key lengths (half of them
at or next to a tile edge: 32, 64, 128, 256, 512 and one either side), the
head dimensions d and d_v, the input dtype, the causal flag, per-batch valid
key lengths and a float32 output, from a fixed seed, so the sweep is the
same on every run.  The shapes reach the decode kernel (few queries), the
4-wave and two-group kernels, key splits, ragged and empty key ranges, and
both sides of the causal kernel switches' tile geometry.  Every output is
held to the same per-tensor and per-row bars as the other parity tests.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_2112_05682_amd import attention_bwd, attention_fwd
from paper_2112_05682_amd.inputs import attention_inputs
from parity_util import TOL, check, check_lse, f64, gradient_row_scales, to_gpu

pytestmark = pytest.mark.gpu

N_CASES = 48
EDGES = [e + o for e in (32, 64, 128, 256, 512) for o in (-1, 0, 1)]


def _length(rng, lo=1, hi=700):
    if rng.random() < 0.5:
        return int(rng.choice(EDGES))
    return int(rng.integers(lo, hi + 1))


def _case(i):
    rng = np.random.default_rng(1000 + i)
    B = int(rng.integers(1, 3))
    H = int(rng.integers(1, 4))
    nq = _length(rng)
    nk = _length(rng)
    d = int(rng.choice([64, 128]))
    d_v = d if rng.random() < 0.8 else 192 - d
    dtype = str(rng.choice(["bf16", "bf16", "fp16", "fp32"]))
    causal = bool(rng.random() < 0.5)
    kv_len = [int(rng.integers(0, nk + 1)) for _ in range(B)] if rng.random() < 0.25 else None
    out_f32 = dtype != "fp32" and rng.random() < 0.15
    return B, H, nq, nk, d, d_v, dtype, causal, kv_len, out_f32


CASES = [_case(i) for i in range(N_CASES)]


def _ids(c):
    B, H, nq, nk, d, d_v, dtype, causal, kv_len, out_f32 = c
    s = "%dx%dx%dx%d-d%d" % (B, H, nq, nk, d) + ("-dv%d" % d_v if d_v != d else "")
    s += "-" + dtype + ("-causal" if causal else "")
    s += ("-kv" + "_".join(map(str, kv_len)) if kv_len else "") + ("-f32o" if out_f32 else "")
    return s


@pytest.mark.parametrize("case", CASES, ids=_ids)
def test_random_problem_matches_oracle(case):
    B, H, nq, nk, d, d_v, dtype, causal, kv_len, out_f32 = case
    print("fuzz case", _ids(case), flush=True)
    x = attention_inputs(B, H, nq, nk, d, dtype, with_grad=True, d_v=d_v,
                         seeds=(zlib.crc32(_ids(case).encode()) % 1000, 11, 12, 13))
    g = to_gpu(x)
    kl = torch.tensor(kv_len, dtype=torch.int32, device="cuda") if kv_len else None
    o, lse, o_lo = attention_fwd(g["q"], g["k"], g["v"], causal=causal, kv_len=kl,
                                 out_dtype=torch.float32 if out_f32 else None, residual=True)
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
    for b in range(B):
        n = nk if kv_len is None else max(0, min(kv_len[b], nk))
        if n == 0:
            # No visible key: o = 0, lse = -inf and zero gradients.
            assert np.all(got["O"][b] == 0.0) and np.all(got["LSE"][b] == -np.inf)
            assert all(np.all(got[k_][b] == 0.0) for k_ in ("dQ", "dK", "dV"))
            continue
        for name in ("O", "dQ", "dK", "dV"):
            check(name, got[name][b], ref[name][b], TOL[dtype], lead=1,
                  terms=terms[name][b] if name in terms else None)
        check_lse(got["LSE"][b], ref["LSE"][b])

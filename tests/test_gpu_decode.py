"""GPU parity of the decode-shaped forward (at most 64 queries per batch and
head, 16-bit inputs) against the float64 oracle.

These shapes run the key-streaming decode kernel: one wave per key range, the
ranges' summaries combined afterwards (Section 4) when there is more than one.
Cases cover one query (the paper's single-query algorithm, Section 2), query
groups on both sides of the 32-query sub-tile, ragged key tiles, one range and
many ranges, causal masking, a float32 output and large logits.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2112_05682_amd import _lib, attention_fwd
from paper_2112_05682_amd.inputs import WORKLOADS, attention_inputs, workload_inputs
from parity_util import TOL, check, check_lse, f64, to_gpu

pytestmark = pytest.mark.gpu

DT = {"bf16": 2, "fp16": 1}


def run_case(B, H, nq, nk, d, dtype, causal=False, out_dtype=None, qk_mult=1.0, seeds=(0, 1, 2, 3)):
    print("decode case B=%d H=%d nq=%d nk=%d d=%d %s causal=%s out=%s mult=%s" % (
        B, H, nq, nk, d, dtype, causal, out_dtype, qk_mult), flush=True)
    x = attention_inputs(B, H, nq, nk, d, dtype, 1.0, qk_mult, seeds, with_grad=False)
    g = to_gpu(x)
    o, lse = attention_fwd(g["q"], g["k"], g["v"], causal=causal, out_dtype=out_dtype)
    torch.cuda.synchronize()
    ro, rl = oracle.fwd(f64(x["q"]), f64(x["k"]), f64(x["v"]), scale=d ** -0.5, causal=causal)
    assert np.all(np.isfinite(f64(lse)))
    check("O", f64(o), ro, TOL[dtype])
    check_lse(f64(lse), rl)


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("nq", [1, 5, 32, 33, 64])
@pytest.mark.parametrize("nk", [1, 31, 65, 1000, 9000])
def test_decode_shapes(dtype, d, nq, nk):
    run_case(2, 3, nq, nk, d, dtype)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("nq", [1, 7, 40, 64])
@pytest.mark.parametrize("nk", [1, 50, 3000])
def test_decode_causal(d, nq, nk):
    # Top-left causal: query i sees keys 0 .. i, so a group of nq queries
    # reads at most the first nq keys.
    run_case(1, 2, nq, nk, d, "bf16", causal=True)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("nq", [3, 48])
def test_decode_many_ranges(d, nq):
    # One (batch, head): the keys are split into many ranges (workspace > 0);
    # 48 queries run two 32-query sub-tiles per wave.
    B, H, nk = 1, 1, 200001
    assert _lib.fwd_workspace_size(_lib.problem(B, H, nq, nk, d, 2, False, d ** -0.5)) > 0
    run_case(B, H, nq, nk, d, "bf16")


def test_decode_one_range_needs_no_workspace():
    # Many (batch, head) pairs and few keys: one range each, no combine.
    assert _lib.fwd_workspace_size(_lib.problem(64, 32, 1, 200, 64, 2, False, 0.125)) == 0
    run_case(64, 32, 1, 200, 64, "bf16")


@pytest.mark.parametrize("dtype", ["bf16", "fp16"])
def test_decode_float32_output(dtype):
    run_case(2, 2, 9, 5000, 64, dtype, out_dtype=torch.float32)


@pytest.mark.parametrize("d", [64, 128])
def test_decode_large_logits(d):
    # Q and K scaled by 30: logits far beyond the float32 exp range.
    run_case(1, 2, 16, 4000, d, "bf16", qk_mult=30.0, out_dtype=torch.float32)


def test_decode_boundary_to_tiled_path():
    # 64 queries take the decode kernel, 65 the query-tiled kernel: both agree
    # with the oracle on the same keys.
    run_case(1, 2, 64, 2000, 64, "bf16")
    run_case(1, 2, 65, 2000, 64, "bf16")


def test_decode_is_deterministic():
    x = to_gpu(attention_inputs(2, 4, 3, 70000, 64, "bf16", with_grad=False))
    o1, l1 = attention_fwd(x["q"], x["k"], x["v"])
    o2, l2 = attention_fwd(x["q"], x["k"], x["v"])
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.parametrize("name", ["decode_bf16_b8h16_nq1_nk65536_d64",
                                  "decode_bf16_b8h16_nq16_nk65536_d64"])
def test_decode_full_size_sampled(name):
    # The decode workloads at full size, in the launch configuration the
    # benchmark uses; the oracle recomputes a few whole (batch, head) slices.
    w = WORKLOADS[name]
    print("workload", name, flush=True)
    x = workload_inputs(w, with_grad=False)
    g = to_gpu(x)
    o, lse = attention_fwd(g["q"], g["k"], g["v"], causal=w.causal)
    torch.cuda.synchronize()
    o_c, l_c = o.cpu(), lse.cpu()
    for b, h in sorted({(0, 0), (w.batch - 1, w.heads - 1), (w.batch // 2, w.heads // 3)}):
        ro, rl = oracle.fwd(f64(x["q"][b, h][None, None]), f64(x["k"][b, h][None, None]),
                            f64(x["v"][b, h][None, None]), scale=w.d ** -0.5, causal=w.causal)
        print("  slice", (b, h), flush=True)
        check("O", f64(o_c[b, h]), ro[0, 0], TOL[w.dtype])
        check_lse(f64(l_c[b, h]), rl[0, 0])
    assert torch.isfinite(o).all() and torch.isfinite(lse).all()


def test_decode_staged_combine_long_keys():
    # 2^22 keys for one (batch, head): 1024 key ranges, combined in three
    # stages of 16 ranges and a final combine (Section 4's combine as a tree).
    B, H, nq, nk, d = 1, 1, 2, 1 << 22, 64
    ws = _lib.fwd_workspace_size(_lib.problem(B, H, nq, nk, d, 2, False, d ** -0.5))
    assert ws > 1024 * nq * (d + 2) * 4  # room for the ranges and the stage buffer
    run_case(B, H, nq, nk, d, "bf16")

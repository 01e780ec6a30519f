"""CPU checks that the parity metrics discriminate (no GPU involved).

A metric that only divides by the whole tensor's largest element cannot see
rows whose values are far smaller than that element; under a causal mask late
rows average thousands of value vectors, so their entries are ~sqrt(i) times
smaller than row 0's (a single value vector).  These tests plant mistakes in
the float64 oracle's own output and show that the per-row metric and the
elementwise lse bar reject them, while legitimate 16-bit rounding passes.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2112_05682_amd.inputs import attention_inputs
from parity_util import TOL, gradient_row_scales, lse_err, rel_err, row_err


@pytest.fixture(scope="module")
def causal_c4_like():
    # The causal d = 128 workload's statistics (N(0, 0.5^2)), one head, n = 4096.
    x = attention_inputs(1, 1, 4096, 4096, 128, "bf16", std=0.5, with_grad=False)
    q, k, v = (x[n].to(torch.float64).numpy() for n in ("q", "k", "v"))
    o, lse = oracle.fwd(q, k, v, scale=128 ** -0.5, causal=True)
    return o, lse


def test_zeroed_late_causal_rows_pass_the_tensor_metric_but_fail_the_row_metric(causal_c4_like):
    o, _ = causal_c4_like
    top = np.abs(o).max()
    row_max = np.abs(o[0, 0]).max(axis=1)
    hidden = np.nonzero(row_max < TOL["bf16"] * top)[0]
    n = o.shape[2]
    # Most of the second half is invisible to the whole-tensor metric ...
    assert np.sum(hidden >= n // 2) > 0.5 * (n // 2)
    bad = o.copy()
    bad[0, 0, hidden] = 0.0
    assert rel_err(bad, o) <= TOL["bf16"]
    # ... and the per-row metric sees every one of those rows.
    assert row_err(bad, o) >= 0.99
    # Zeroing a single late row is caught too.
    one = o.copy()
    one[0, 0, n - 1] = 0.0
    assert row_err(one, o) >= 0.99


def test_row_metric_accepts_16_bit_rounding(causal_c4_like):
    o, _ = causal_c4_like
    for dt in (torch.bfloat16, torch.float16):
        r = torch.from_numpy(o).to(dt).to(torch.float64).numpy()
        assert row_err(r, o) <= 2.0 ** -8  # one rounding: at most half an ulp relative


def test_row_metric_floor_ignores_rows_that_are_exactly_zero_in_the_reference():
    # A row whose reference is 0 (e.g. dK of a padded key) is measured against
    # 1e-3 of the tensor's largest element, not against 0.
    ref = np.array([[1.0, -2.0], [0.0, 0.0]])
    got = np.array([[1.0, -2.0], [1e-5, 0.0]])
    assert row_err(got, ref) == pytest.approx(1e-5 / 2e-3)


def test_lse_bar_is_elementwise_and_tight(causal_c4_like):
    _, lse = causal_c4_like
    f32 = lse.astype(np.float32).astype(np.float64)
    assert lse_err(f32, lse) <= 0.01  # float32 rounding of the value itself
    shifted = lse.copy()
    shifted[0, 0, -1] += 1e-3  # one late row off by 1e-3 nats
    assert lse_err(shifted, lse) > 1.0
    # The old whole-tensor metric (2e-2 of max|lse|) would have accepted 0.1 nats.
    off = lse.copy()
    off[0, 0, -1] += 0.1
    assert rel_err(off, lse) <= TOL["bf16"]
    assert lse_err(off, lse) > 1.0


def test_lse_bar_treats_matching_minus_infinity_as_exact():
    ref = np.array([-np.inf, 3.0])
    assert lse_err(np.array([-np.inf, 3.0]), ref) == 0.0
    assert lse_err(np.array([0.0, 3.0]), ref) == np.inf


@pytest.mark.parametrize("causal,kv_len", [(False, None), (True, None), (True, [9, 4])])
def test_gradient_row_scales_bound_the_reference(causal, kv_len):
    # |dQ_if| <= scale sum_j P_ij (|dP_ij| + |D_i|) |k_jf| <= cq_i (triangle
    # inequality, twice), and likewise for dK: the scale is never below the value.
    x = attention_inputs(2, 2, 11, 13, 8, "fp32", with_grad=True)
    q, k, v, do = (x[n].to(torch.float64).numpy() for n in ("q", "k", "v", "do"))
    _, lse = oracle.fwd(q, k, v, scale=0.3, causal=causal, kv_len=kv_len)
    rq, rk, _ = oracle.bwd(q, k, v, do, scale=0.3, causal=causal, kv_len=kv_len)
    cq, ck = gradient_row_scales(q, k, v, do, lse, 0.3, causal, kv_len)
    assert np.all(np.abs(rq).max(axis=-1) <= cq * (1 + 1e-12) + 1e-300)
    assert np.all(np.abs(rk).max(axis=-1) <= ck * (1 + 1e-12) + 1e-300)
    # Causal row 0 of dQ is an exact cancellation (one visible key): value 0,
    # scale not 0.
    if causal:
        assert np.abs(rq[:, :, 0]).max() < 1e-12 and cq[:, :, 0].min() > 0.1


def test_zeroed_late_gradient_rows_are_caught_with_term_scales():
    # The widened scale of dQ / dK rows still rejects a row replaced by zeros.
    x = attention_inputs(1, 1, 2048, 2048, 128, "bf16", std=0.5, with_grad=True)
    q, k, v, do = (x[n].to(torch.float64).numpy() for n in ("q", "k", "v", "do"))
    s = 128 ** -0.5
    _, lse = oracle.fwd(q, k, v, scale=s, causal=True)
    rq, rk, _ = oracle.bwd(q, k, v, do, scale=s, causal=True)
    cq, ck = gradient_row_scales(q, k, v, do, lse, s, True)
    for ref, terms in ((rq, cq), (rk, ck)):
        for row in (1, 700, 2046):
            bad = ref.copy()
            bad[0, 0, row] = 0.0
            assert row_err(bad, ref, terms=terms) > TOL["bf16"], row
        r16 = torch.from_numpy(ref).to(torch.bfloat16).to(torch.float64).numpy()
        assert row_err(r16, ref, terms=terms) <= 2.0 ** -8

"""Seeded fuzz of the float64 oracle on tiny problems (CPU only).

Random shapes (batch, heads, n_q, n_k, d, d_v), masks (causal, per-batch
valid key lengths including empty batches), logit magnitudes up to ~1e3 and
chunk sizes; hypothesis runs derandomized, so every run draws the same cases.

* The three forward forms -- the Section 1 definition, the Section 3 running
  update and the Section 4 chunk summaries -- agree to ~1e-12.
* The hand-derived backward agrees with central finite differences of
  L = sum(dO * O) for every element of q, k and v.
"""
import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle

SETTINGS = dict(deadline=None, derandomize=True, suppress_health_check=[HealthCheck.too_slow])


@st.composite
def problems(draw, max_n=9, max_d=6):
    B = draw(st.integers(1, 2))
    H = draw(st.integers(1, 2))
    nq = draw(st.integers(1, max_n))
    nk = draw(st.integers(1, max_n))
    d = draw(st.integers(1, max_d))
    dv = draw(st.integers(1, max_d))
    causal = draw(st.booleans())
    kv_len = draw(st.one_of(st.none(), st.lists(st.integers(-1, nk + 2), min_size=B, max_size=B)))
    seed = draw(st.integers(0, 2 ** 31 - 1))
    return B, H, nq, nk, d, dv, causal, kv_len, seed


def _inputs(B, H, nq, nk, d, dv, seed, amp):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, H, nq, d)) * amp
    k = rng.standard_normal((B, H, nk, d)) * amp
    v = rng.standard_normal((B, H, nk, dv))
    do = rng.standard_normal((B, H, nq, dv))
    return q, k, v, do


def _close(a, b, tol):
    a, b = np.asarray(a), np.asarray(b)
    same_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    a = np.where(same_inf, 0.0, a)
    b = np.where(same_inf, 0.0, b)
    top = max(np.abs(b).max(initial=0.0), 1e-300)
    return np.abs(a - b).max(initial=0.0) <= tol * max(top, 1.0)


@settings(max_examples=300, **SETTINGS)
@given(problems(), st.sampled_from([0.1, 1.0, 10.0, 40.0]), st.integers(1, 12), st.integers(1, 12))
def test_three_forward_forms_agree(prob, amp, qc, kc):
    B, H, nq, nk, d, dv, causal, kv_len, seed = prob
    q, k, v, _ = _inputs(B, H, nq, nk, d, dv, seed, amp)
    o1, l1 = oracle.fwd(q, k, v, causal=causal, kv_len=kv_len)
    o2, l2 = oracle.fwd_lazy(q, k, v, causal=causal, kv_len=kv_len)
    o3, l3 = oracle.fwd_chunked(q, k, v, causal=causal, query_chunk=qc, key_chunk=kc, kv_len=kv_len)
    assert np.all(np.isfinite(o1))
    for o, lse in ((o2, l2), (o3, l3)):
        assert _close(o, o1, 1e-12)
        assert _close(lse, l1, 1e-12)


@settings(max_examples=60, **SETTINGS)
@given(problems(max_n=5, max_d=3), st.sampled_from([0.3, 1.0, 2.0]))
def test_backward_matches_central_differences(prob, amp):
    B, H, nq, nk, d, dv, causal, kv_len, seed = prob
    q, k, v, do = _inputs(B, H, nq, nk, d, dv, seed, amp)
    dq, dk, dv_ = oracle.bwd(q, k, v, do, causal=causal, kv_len=kv_len)

    def loss(q_, k_, v_):
        o, _ = oracle.fwd(q_, k_, v_, causal=causal, kv_len=kv_len)
        return float((o * do).sum())

    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv_)):
        fd = np.zeros_like(x)
        for idx in np.ndindex(*x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = {"q": q, "k": k, "v": v}
            args_m = dict(args_p)
            args_p[name], args_m[name] = xp, xm
            fd[idx] = (loss(**{n_ + "_": a for n_, a in args_p.items()}) -
                       loss(**{n_ + "_": a for n_, a in args_m.items()})) / (2 * h)
        scale = max(np.abs(g).max(initial=0.0), 1.0)
        err = np.abs(fd - g).max(initial=0.0) / scale
        assert err <= 2e-6, (name, err)


@pytest.mark.parametrize("amp", [300.0])
def test_forward_forms_agree_at_logits_of_order_1e4(amp):
    # Far beyond the float64 exp overflow at ~709 (the Section 3 setting).
    q, k, v, _ = _inputs(1, 2, 7, 11, 4, 3, 123, amp)
    o1, l1 = oracle.fwd(q, k, v, causal=True)
    o2, l2 = oracle.fwd_lazy(q, k, v, causal=True)
    o3, l3 = oracle.fwd_chunked(q, k, v, causal=True, query_chunk=2, key_chunk=3)
    assert np.all(np.isfinite(o1)) and np.all(np.isfinite(l1))
    assert _close(o2, o1, 1e-12) and _close(o3, o1, 1e-12)
    assert _close(l2, l1, 1e-12) and _close(l3, l1, 1e-12)

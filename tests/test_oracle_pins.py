"""Pins for the float64 CPU oracle (CPU only, no GPU).

The oracle must be right before anything is compared with it, so every
function in it is checked here against facts that do not come from the oracle
itself: a hand-derived worked example, closed forms, invariants of softmax
attention, library routines (scipy's softmax / logsumexp), finite
differences of the forward, and the overflow fact of the paper's Section 3.
"""
import math
import os

import numpy as np
import pytest
from scipy.special import logsumexp, softmax

FORWARD_FORMS = ("direct", "lazy", "chunked")
GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "two_key_example.txt")


def run_fwd(oracle, form, q, k, v, scale=None, causal=False, key_chunk=3, query_chunk=2):
    if form == "direct":
        return oracle.fwd(q, k, v, scale, causal)
    if form == "lazy":
        return oracle.fwd_lazy(q, k, v, scale, causal)
    return oracle.fwd_chunked(q, k, v, scale, causal, query_chunk=query_chunk,
                              key_chunk=key_chunk)


def rand(shape, seed, std=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * std


def read_golden():
    vals = {}
    env = {"ln3": math.log(3.0), "ln4": math.log(4.0)}
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, rhs = (s.strip() for s in line.split("=", 1))
            vals[name] = np.array([eval(tok, {"__builtins__": {}}, env)
                                   for tok in rhs.split(",")], dtype=np.float64)
    return vals


# ---------------------------------------------------------------- worked example

@pytest.mark.parametrize("form", FORWARD_FORMS)
def test_golden_two_key_forward(oracle_mod, form):
    g = read_golden()
    q = g["q"].reshape(1, 1, 1, 2)
    k = g["k"].reshape(1, 1, 2, 2)
    v = g["v"].reshape(1, 1, 2, 2)
    o, lse = run_fwd(oracle_mod, form, q, k, v, scale=1.0, key_chunk=1, query_chunk=1)
    np.testing.assert_allclose(o.ravel(), g["o"], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(lse.ravel(), g["lse"], rtol=1e-14)


def test_golden_two_key_backward(oracle_mod):
    g = read_golden()
    q = g["q"].reshape(1, 1, 1, 2)
    k = g["k"].reshape(1, 1, 2, 2)
    v = g["v"].reshape(1, 1, 2, 2)
    do = g["do"].reshape(1, 1, 1, 2)
    dq, dk, dv = oracle_mod.bwd(q, k, v, do, scale=1.0)
    np.testing.assert_allclose(dq.ravel(), g["dq"], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(dk.ravel(), g["dk"], rtol=1e-14, atol=1e-14)
    np.testing.assert_allclose(dv.ravel(), g["dv"], rtol=1e-14, atol=1e-14)


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("form", FORWARD_FORMS)
@pytest.mark.parametrize("causal", [False, True])
def test_zero_query_gives_mean_of_visible_values(oracle_mod, form, causal):
    # Q = 0 makes every score 0: the weights are uniform over the visible keys.
    B, H, nq, nk, d = 2, 2, 6, 9, 5
    q = np.zeros((B, H, nq, d))
    k = rand((B, H, nk, d), 1)
    v = rand((B, H, nk, d), 2)
    o, lse = run_fwd(oracle_mod, form, q, k, v, causal=causal)
    for i in range(nq):
        n_vis = min(i + 1, nk) if causal else nk
        np.testing.assert_allclose(o[:, :, i], v[:, :, :n_vis].mean(axis=2), rtol=1e-13,
                                   atol=1e-14)
        np.testing.assert_allclose(lse[:, :, i], math.log(n_vis), rtol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_zero_query_gradients(oracle_mod, causal):
    # Uniform weights: dS_ij = w (dO_i.v_j - mean_j dO_i.v_j), dK = scale * dS^T Q = 0,
    # dV_j = sum over queries that see j of dO_i / |J(i)|.
    B, H, nq, nk, d = 1, 2, 6, 9, 4
    q = np.zeros((B, H, nq, d))
    k, v, do = rand((B, H, nk, d), 3), rand((B, H, nk, d), 4), rand((B, H, nq, d), 5)
    dq, dk, dv = oracle_mod.bwd(q, k, v, do, causal=causal)
    np.testing.assert_allclose(dk, 0.0, atol=1e-15)
    expect = np.zeros_like(v)
    for i in range(nq):
        n_vis = min(i + 1, nk) if causal else nk
        expect[:, :, :n_vis] += do[:, :, i:i + 1] / n_vis
    np.testing.assert_allclose(dv, expect, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("form", FORWARD_FORMS)
def test_single_key(oracle_mod, form):
    # n_k = 1: the only weight is 1, o = v_0 and lse = s_0.
    B, H, nq, d = 1, 3, 5, 4
    q, k, v = rand((B, H, nq, d), 6), rand((B, H, 1, d), 7), rand((B, H, 1, d), 8)
    scale = 0.7
    o, lse = run_fwd(oracle_mod, form, q, k, v, scale=scale)
    np.testing.assert_allclose(o, np.broadcast_to(v, o.shape), rtol=1e-14)
    s0 = scale * np.einsum("bhid,bhjd->bhi", q, k)
    np.testing.assert_allclose(lse, s0, rtol=1e-14, atol=1e-15)


def test_single_key_gradients(oracle_mod):
    B, H, nq, d = 1, 2, 5, 4
    q, k, v, do = (rand((B, H, nq, d), 9), rand((B, H, 1, d), 10), rand((B, H, 1, d), 11),
                   rand((B, H, nq, d), 12))
    dq, dk, dv = oracle_mod.bwd(q, k, v, do)
    np.testing.assert_allclose(dq, 0.0, atol=1e-15)
    np.testing.assert_allclose(dk, 0.0, atol=1e-15)
    np.testing.assert_allclose(dv[:, :, 0], do.sum(axis=2), rtol=1e-14)


@pytest.mark.parametrize("form", FORWARD_FORMS)
def test_dominant_key_returns_its_value(oracle_mod, form):
    # A key parallel to the query whose score beats every other by >= 50
    # carries weight 1 - O(n e^-50).
    d, nk, j_star, scale = 8, 33, 17, 0.5
    q = rand((1, 1, 1, d), 13)
    k = rand((1, 1, nk, d), 14, std=0.1)
    v = rand((1, 1, nk, d), 15)
    others = scale * np.einsum("d,jd->j", q[0, 0, 0], k[0, 0])
    target = others.max() + 60.0
    k[0, 0, j_star] = q[0, 0, 0] * target / (scale * float(q[0, 0, 0] @ q[0, 0, 0]))
    o, lse = run_fwd(oracle_mod, form, q, k, v, scale=scale, key_chunk=5)
    bound = nk * math.exp(-50.0) * np.abs(v).max()
    assert np.abs(o[0, 0, 0] - v[0, 0, j_star]).max() <= bound
    # the constructed score equals `target` only up to rounding of k_{j*}
    assert abs(lse[0, 0, 0] - target) <= nk * math.exp(-50.0) + 1e-13 * target


# ---------------------------------------------------------------- library routines

@pytest.mark.parametrize("form", FORWARD_FORMS)
@pytest.mark.parametrize("causal", [False, True])
def test_matches_scipy_softmax(oracle_mod, form, causal):
    B, H, nq, nk, d = 2, 3, 7, 11, 5
    q, k, v = rand((B, H, nq, d), 16), rand((B, H, nk, d), 17), rand((B, H, nk, d), 18)
    scale = 0.37
    o, lse = run_fwd(oracle_mod, form, q, k, v, scale=scale, causal=causal)
    for b in range(B):
        for h in range(H):
            s = scale * (q[b, h] @ k[b, h].T)
            if causal:
                s = np.where(np.arange(nk)[None, :] <= np.arange(nq)[:, None], s, -np.inf)
            np.testing.assert_allclose(o[b, h], softmax(s, axis=1) @ v[b, h], rtol=1e-12,
                                       atol=1e-13)
            np.testing.assert_allclose(lse[b, h], logsumexp(s, axis=1), rtol=1e-13)


# ---------------------------------------------------------------- invariants

@pytest.mark.parametrize("form", FORWARD_FORMS)
def test_joint_key_value_permutation(oracle_mod, form):
    B, H, nq, nk, d = 1, 2, 5, 10, 4
    q, k, v, do = (rand((B, H, nq, d), 19), rand((B, H, nk, d), 20), rand((B, H, nk, d), 21),
                   rand((B, H, nq, d), 22))
    perm = np.random.default_rng(23).permutation(nk)
    o1, l1 = run_fwd(oracle_mod, form, q, k, v)
    o2, l2 = run_fwd(oracle_mod, form, q, k[:, :, perm], v[:, :, perm])
    np.testing.assert_allclose(o2, o1, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(l2, l1, rtol=1e-13)
    if form == "direct":
        dq1, dk1, dv1 = oracle_mod.bwd(q, k, v, do)
        dq2, dk2, dv2 = oracle_mod.bwd(q, k[:, :, perm], v[:, :, perm], do)
        np.testing.assert_allclose(dq2, dq1, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(dk2, dk1[:, :, perm], rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(dv2, dv1[:, :, perm], rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("form", FORWARD_FORMS)
@pytest.mark.parametrize("causal", [False, True])
def test_value_shift(oracle_mod, form, causal):
    # Weights sum to one, so adding c to every value adds c to every output.
    B, H, nq, nk, d = 1, 2, 6, 8, 3
    q, k, v = rand((B, H, nq, d), 24), rand((B, H, nk, d), 25), rand((B, H, nk, d), 26)
    c = np.array([3.0, -2.0, 0.5])
    o1, _ = run_fwd(oracle_mod, form, q, k, v, causal=causal)
    o2, _ = run_fwd(oracle_mod, form, q, k, v + c, causal=causal)
    np.testing.assert_allclose(o2, o1 + c, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_key_shift(oracle_mod, causal):
    # Adding u to every key adds scale*q_i.u to every score of row i: O and all
    # gradients are unchanged, lse moves by scale*q_i.u.
    B, H, nq, nk, d = 1, 2, 6, 8, 3
    q, k, v, do = (rand((B, H, nq, d), 27), rand((B, H, nk, d), 28), rand((B, H, nk, d), 29),
                   rand((B, H, nq, d), 30))
    u = np.array([1.5, -0.25, 2.0])
    scale = 0.8
    o1, l1 = oracle_mod.fwd(q, k, v, scale, causal)
    o2, l2 = oracle_mod.fwd(q, k + u, v, scale, causal)
    np.testing.assert_allclose(o2, o1, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l2, l1 + scale * (q @ u), rtol=1e-12, atol=1e-13)
    g1 = oracle_mod.bwd(q, k, v, do, scale, causal)
    g2 = oracle_mod.bwd(q, k + u, v, do, scale, causal)
    for a, b in zip(g1, g2):
        np.testing.assert_allclose(b, a, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_gradient_sum_rules(oracle_mod, causal):
    # Each dS row sums to zero, so sum_j dK_j = 0; each weight row sums to one,
    # so sum_j dV_j = sum_i dO_i.
    B, H, nq, nk, d = 2, 2, 9, 7, 4
    q, k, v, do = (rand((B, H, nq, d), 31), rand((B, H, nk, d), 32), rand((B, H, nk, d), 33),
                   rand((B, H, nq, d), 34))
    dq, dk, dv = oracle_mod.bwd(q, k, v, do, causal=causal)
    np.testing.assert_allclose(dk.sum(axis=2), 0.0, atol=1e-13)
    np.testing.assert_allclose(dv.sum(axis=2), do.sum(axis=2), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("form", FORWARD_FORMS)
def test_causal_row_is_attention_over_its_prefix(oracle_mod, form):
    # Under the top-left causal reading, row i of a causal call equals the
    # unmasked attention of query i over keys 0..i (and over all keys when
    # i >= n_k).
    B, H, nq, nk, d = 1, 1, 9, 6, 4
    q, k, v = rand((B, H, nq, d), 35), rand((B, H, nk, d), 36), rand((B, H, nk, d), 37)
    o, lse = run_fwd(oracle_mod, form, q, k, v, causal=True)
    for i in range(nq):
        n_vis = min(i + 1, nk)
        oi, li = run_fwd(oracle_mod, form, q[:, :, i:i + 1], k[:, :, :n_vis], v[:, :, :n_vis])
        np.testing.assert_allclose(o[:, :, i:i + 1], oi, rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(lse[:, :, i:i + 1], li, rtol=1e-14)


def test_causal_gradients_match_prefix_problems(oracle_mod):
    # The causal loss is a sum of per-row prefix losses, so its gradients are
    # the sum of the prefix problems' gradients.
    B, H, nq, nk, d = 1, 1, 6, 6, 3
    q, k, v, do = (rand((B, H, nq, d), 38), rand((B, H, nk, d), 39), rand((B, H, nk, d), 40),
                   rand((B, H, nq, d), 41))
    dq, dk, dv = oracle_mod.bwd(q, k, v, do, causal=True)
    edq, edk, edv = np.zeros_like(dq), np.zeros_like(dk), np.zeros_like(dv)
    for i in range(nq):
        n = i + 1
        a, b_, c = oracle_mod.bwd(q[:, :, i:i + 1], k[:, :, :n], v[:, :, :n], do[:, :, i:i + 1])
        edq[:, :, i:i + 1] += a
        edk[:, :, :n] += b_
        edv[:, :, :n] += c
    for got, exp in ((dq, edq), (dk, edk), (dv, edv)):
        np.testing.assert_allclose(got, exp, rtol=1e-12, atol=1e-14)


# ---------------------------------------------------------------- forms agree

@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("shape", [(1, 1, 1, 1, 1), (1, 2, 7, 13, 5), (2, 1, 13, 7, 3),
                                   (1, 1, 33, 100, 8)])
def test_three_forward_forms_agree(oracle_mod, causal, shape):
    B, H, nq, nk, d = shape
    q, k, v = rand((B, H, nq, d), 42), rand((B, H, nk, d), 43), rand((B, H, nk, d), 44)
    o0, l0 = oracle_mod.fwd(q, k, v, causal=causal)
    o1, l1 = oracle_mod.fwd_lazy(q, k, v, causal=causal)
    np.testing.assert_allclose(o1, o0, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l1, l0, rtol=1e-13, atol=1e-14)
    for kc, qc in ((1, 1), (3, 2), (4, 5), (nk, nq), (nk + 5, 1000)):
        o2, l2 = oracle_mod.fwd_chunked(q, k, v, causal=causal, query_chunk=qc, key_chunk=kc)
        np.testing.assert_allclose(o2, o0, rtol=1e-12, atol=1e-13)
        np.testing.assert_allclose(l2, l0, rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------- finite differences

@pytest.mark.parametrize("causal", [False, True])
def test_gradients_match_central_differences(oracle_mod, causal):
    B, H, nq, nk, d = 1, 2, 5, 7, 3
    q, k, v, do = (rand((B, H, nq, d), 45), rand((B, H, nk, d), 46), rand((B, H, nk, d), 47),
                   rand((B, H, nq, d), 48))
    scale = 0.9

    def loss(q_, k_, v_):
        o, _ = oracle_mod.fwd(q_, k_, v_, scale, causal)
        return float((o * do).sum())

    dq, dk, dv = oracle_mod.bwd(q, k, v, do, scale, causal)
    h = 1e-6
    for which, grad in ((0, dq), (1, dk), (2, dv)):
        args = [q, k, v]
        base = args[which]
        fd = np.zeros_like(base)
        for idx in np.ndindex(base.shape):
            plus = base.copy()
            minus = base.copy()
            plus[idx] += h
            minus[idx] -= h
            a_p = list(args)
            a_m = list(args)
            a_p[which] = plus
            a_m[which] = minus
            fd[idx] = (loss(*a_p) - loss(*a_m)) / (2 * h)
        err = np.abs(fd - grad).max() / max(np.abs(grad).max(), 1e-300)
        assert err < 1e-7, (which, err)


# ---------------------------------------------------------------- subsets

def test_row_and_key_subsets_match_full(oracle_mod):
    nq, nk, d = 37, 29, 6
    q, k, v, do = (rand((nq, d), 49), rand((nk, d), 50), rand((nk, d), 51), rand((nq, d), 52))
    for causal in (False, True):
        o, lse = oracle_mod.fwd(q[None, None], k[None, None], v[None, None], causal=causal)
        dq, dk, dv = oracle_mod.bwd(q[None, None], k[None, None], v[None, None], do[None, None],
                                    causal=causal)
        rows = np.array([36, 0, 17, 5, 5])
        orow, lrow = oracle_mod.fwd_rows(q, k, v, rows, causal=causal)
        np.testing.assert_array_equal(orow, o[0, 0, rows])
        np.testing.assert_array_equal(lrow, lse[0, 0, rows])
        np.testing.assert_array_equal(oracle_mod.bwd_dq_rows(q, k, v, do, rows, causal=causal),
                                      dq[0, 0, rows])
        keys = np.array([28, 3, 0, 11])
        dkr, dvr = oracle_mod.bwd_dkdv_keys(q, k, v, do, keys, causal=causal)
        np.testing.assert_array_equal(dkr, dk[0, 0, keys])
        np.testing.assert_array_equal(dvr, dv[0, 0, keys])


def test_invalid_arguments_raise(oracle_mod):
    q = np.zeros((4, 2))
    with pytest.raises(RuntimeError):
        oracle_mod.fwd_rows(q, q, q, [4])
    with pytest.raises(RuntimeError):
        oracle_mod.bwd_dkdv_keys(q, q, q, q, [-1])
    with pytest.raises(RuntimeError):
        oracle_mod.fwd_chunked(q[None, None], q[None, None], q[None, None], key_chunk=0)


# ---------------------------------------------------------------- overflow (Section 3)

def test_exp_overflow_threshold_float32():
    # Section 3: exponentiating scores >= 89 overflows in float32 (ln of the
    # largest float32 is about 88.72).
    with np.errstate(over="ignore"):
        assert np.isinf(np.exp(np.float32(89.0)))
    assert np.isfinite(np.exp(np.float32(88.0)))
    assert 88.0 < math.log(np.finfo(np.float32).max) < 89.0


def _softmax_attention_without_max_subtraction_f32(q, k, v, scale):
    # Deliberately naive float32 helper (test only): the unstable formulation
    # that the paper's Section 3 warns about.
    s = (scale * (q @ k.T)).astype(np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        e = np.exp(s)
        return (e @ v.astype(np.float32)) / e.sum(axis=1, keepdims=True)


@pytest.mark.parametrize("form", FORWARD_FORMS)
def test_large_logits_stay_finite_and_shift_invariant(oracle_mod, form):
    # Scores near 1e3 (beyond float64's exp range too): the naive float32 form
    # blows up, the oracle's max-subtracted forms stay finite and equal the
    # result for the same scores shifted down to O(1).
    nq, nk, d, scale = 4, 9, 4, 1.0
    rng = np.random.default_rng(53)
    q = rng.standard_normal((nq, d))
    k = rng.standard_normal((nk, d))
    v = rng.standard_normal((nk, d))
    u = np.linalg.lstsq(q, np.full(nq, 1000.0), rcond=None)[0]  # q_i . u = 1000
    k_big = k + u
    naive = _softmax_attention_without_max_subtraction_f32(q, k_big, v, scale)
    assert not np.all(np.isfinite(naive))
    o_big, l_big = run_fwd(oracle_mod, form, q[None, None], k_big[None, None], v[None, None],
                           scale=scale)
    o_ref, l_ref = run_fwd(oracle_mod, form, q[None, None], k[None, None], v[None, None],
                           scale=scale)
    assert np.all(np.isfinite(o_big)) and np.all(np.isfinite(l_big))
    np.testing.assert_allclose(o_big, o_ref, rtol=1e-9, atol=1e-10)
    np.testing.assert_allclose(l_big - 1000.0 * scale, l_ref, rtol=1e-9, atol=1e-9)


# ---------------------------------------------------------------- key padding
# Batch b sees only keys j < kv_len[b] (on top of the causal mask); a row that
# sees no key has o = 0, lse = -inf and zero gradients.  Pinned against scipy
# with -inf scores, closed forms, invariance under changing the padded rows,
# the empty batch, and central differences.

def _masked_scores(q, k, scale, n_valid, causal):
    s = scale * (q @ k.T)
    nq, nk = s.shape
    vis = np.arange(nk)[None, :] < n_valid
    if causal:
        vis = vis & (np.arange(nk)[None, :] <= np.arange(nq)[:, None])
    return np.where(vis, s, -np.inf)


def run_fwd_kv(oracle, form, q, k, v, scale, causal, kv_len):
    if form == "direct":
        return oracle.fwd(q, k, v, scale, causal, kv_len=kv_len)
    if form == "lazy":
        return oracle.fwd_lazy(q, k, v, scale, causal, kv_len=kv_len)
    return oracle.fwd_chunked(q, k, v, scale, causal, query_chunk=2, key_chunk=3, kv_len=kv_len)


@pytest.mark.parametrize("form", FORWARD_FORMS)
@pytest.mark.parametrize("causal", [False, True])
def test_key_padding_matches_scipy_softmax(oracle_mod, form, causal):
    B, H, nq, nk, d = 3, 2, 7, 11, 5
    q, k, v = rand((B, H, nq, d), 60), rand((B, H, nk, d), 61), rand((B, H, nk, d), 62)
    kv_len = [4, 11, 1]
    scale = 0.41
    o, lse = run_fwd_kv(oracle_mod, form, q, k, v, scale, causal, kv_len)
    for b in range(B):
        for h in range(H):
            s = _masked_scores(q[b, h], k[b, h], scale, kv_len[b], causal)
            np.testing.assert_allclose(o[b, h], softmax(s, axis=1) @ v[b, h], rtol=1e-12,
                                       atol=1e-13)
            np.testing.assert_allclose(lse[b, h], logsumexp(s, axis=1), rtol=1e-13)


@pytest.mark.parametrize("form", FORWARD_FORMS)
@pytest.mark.parametrize("causal", [False, True])
def test_key_padding_zero_query(oracle_mod, form, causal):
    # Uniform scores: o_i is the mean of the values row i sees, lse_i = ln |J(i)|.
    B, H, nq, nk, d = 2, 1, 6, 9, 3
    v = rand((B, H, nk, d), 63)
    q, k = np.zeros((B, H, nq, d)), rand((B, H, nk, d), 64)
    kv_len = [5, 2]
    o, lse = run_fwd_kv(oracle_mod, form, q, k, v, 0.5, causal, kv_len)
    for b in range(B):
        for i in range(nq):
            n = min(kv_len[b], i + 1) if causal else kv_len[b]
            np.testing.assert_allclose(o[b, 0, i], v[b, 0, :n].mean(axis=0), rtol=1e-13,
                                       atol=1e-14)
            np.testing.assert_allclose(lse[b, 0, i], math.log(n), rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("causal", [False, True])
def test_key_padding_zero_query_gradients(oracle_mod, causal):
    # Q = 0: dK = 0 everywhere, dV_j = sum over the rows that see key j of
    # dO_i / |J(i)|, and padded keys get dV = 0.
    B, H, nq, nk, d = 2, 1, 6, 8, 3
    q, k, v, do = (np.zeros((B, H, nq, d)), rand((B, H, nk, d), 65), rand((B, H, nk, d), 66),
                   rand((B, H, nq, d), 67))
    kv_len = [3, 8]
    dq, dk, dv = oracle_mod.bwd(q, k, v, do, 0.7, causal, kv_len=kv_len)
    np.testing.assert_allclose(dk, 0.0, atol=1e-14)
    for b in range(B):
        want = np.zeros((nk, d))
        for i in range(nq):
            n = min(kv_len[b], i + 1) if causal else kv_len[b]
            want[:n] += do[b, 0, i] / n
        np.testing.assert_allclose(dv[b, 0], want, rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_key_padding_ignores_padded_rows(oracle_mod, causal):
    # Changing k and v at padded positions changes nothing, and the padded
    # keys' gradients are exactly zero.
    B, H, nq, nk, d = 2, 2, 9, 13, 4
    q, k, v, do = (rand((B, H, nq, d), 68), rand((B, H, nk, d), 69), rand((B, H, nk, d), 70),
                   rand((B, H, nq, d), 71))
    kv_len = [6, 10]
    k2, v2 = k.copy(), v.copy()
    for b, n in enumerate(kv_len):
        k2[b, :, n:] = rand(k2[b, :, n:].shape, 72 + b) * 50.0
        v2[b, :, n:] = rand(v2[b, :, n:].shape, 74 + b) * 50.0
    o1, l1 = oracle_mod.fwd(q, k, v, 0.5, causal, kv_len=kv_len)
    o2, l2 = oracle_mod.fwd(q, k2, v2, 0.5, causal, kv_len=kv_len)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(l1, l2)
    g1 = oracle_mod.bwd(q, k, v, do, 0.5, causal, kv_len=kv_len)
    g2 = oracle_mod.bwd(q, k2, v2, do, 0.5, causal, kv_len=kv_len)
    for a, b_ in zip(g1, g2):
        for b, n in enumerate(kv_len):
            np.testing.assert_array_equal(a[b, :, :n] if a.shape[2] == nk else a[b],
                                          b_[b, :, :n] if b_.shape[2] == nk else b_[b])
    for g in (g1[1], g1[2], g2[1], g2[2]):
        for b, n in enumerate(kv_len):
            assert np.all(g[b, :, n:] == 0.0)


@pytest.mark.parametrize("form", FORWARD_FORMS)
def test_key_padding_empty_batch(oracle_mod, form):
    # kv_len = 0: every row of the batch sees no key (o = 0, lse = -inf, zero
    # gradients); the other batch is unaffected.  Negative lengths clamp to 0
    # and lengths past n_k to n_k.
    B, H, nq, nk, d = 2, 2, 4, 6, 3
    q, k, v, do = (rand((B, H, nq, d), 76), rand((B, H, nk, d), 77), rand((B, H, nk, d), 78),
                   rand((B, H, nq, d), 79))
    for lens in ([0, 6], [-3, 99]):
        o, lse = run_fwd_kv(oracle_mod, form, q, k, v, 0.6, False, lens)
        assert np.all(o[0] == 0.0) and np.all(lse[0] == -np.inf)
        o_ref, l_ref = oracle_mod.fwd(q[1:], k[1:], v[1:], 0.6, False)
        np.testing.assert_allclose(o[1], o_ref[0], rtol=1e-13, atol=1e-14)
        np.testing.assert_allclose(lse[1], l_ref[0], rtol=1e-13)
    dq, dk, dv = oracle_mod.bwd(q, k, v, do, 0.6, False, kv_len=[0, 6])
    assert np.all(dq[0] == 0.0) and np.all(dk[0] == 0.0) and np.all(dv[0] == 0.0)


@pytest.mark.parametrize("causal", [False, True])
def test_key_padding_gradients_match_central_differences(oracle_mod, causal):
    B, H, nq, nk, d = 2, 1, 5, 7, 3
    q, k, v, do = (rand((B, H, nq, d), 80), rand((B, H, nk, d), 81), rand((B, H, nk, d), 82),
                   rand((B, H, nq, d), 83))
    scale, kv_len = 0.9, [4, 6]

    def loss(q_, k_, v_):
        o, _ = oracle_mod.fwd(q_, k_, v_, scale, causal, kv_len=kv_len)
        return float((o * do).sum())

    grads = oracle_mod.bwd(q, k, v, do, scale, causal, kv_len=kv_len)
    h = 1e-6
    for which, grad in enumerate(grads):
        args = [q, k, v]
        fd = np.zeros_like(args[which])
        for idx in np.ndindex(fd.shape):
            a_p, a_m = list(args), list(args)
            a_p[which] = args[which].copy()
            a_m[which] = args[which].copy()
            a_p[which][idx] += h
            a_m[which][idx] -= h
            fd[idx] = (loss(*a_p) - loss(*a_m)) / (2 * h)
        err = np.abs(fd - grad).max() / max(np.abs(grad).max(), 1e-300)
        assert err < 1e-7, (which, err)


def test_key_padding_subsets_match_full(oracle_mod):
    nq, nk, d, n_valid = 21, 17, 4, 9
    q, k, v, do = (rand((nq, d), 84), rand((nk, d), 85), rand((nk, d), 86), rand((nq, d), 87))
    for causal in (False, True):
        o, lse = oracle_mod.fwd(q[None, None], k[None, None], v[None, None], causal=causal,
                                kv_len=[n_valid])
        dq, dk, dv = oracle_mod.bwd(q[None, None], k[None, None], v[None, None], do[None, None],
                                    causal=causal, kv_len=[n_valid])
        rows, keys = np.array([20, 0, 8, 3]), np.array([16, 8, 9, 0])
        orow, lrow = oracle_mod.fwd_rows(q, k, v, rows, causal=causal, n_valid=n_valid)
        np.testing.assert_array_equal(orow, o[0, 0, rows])
        np.testing.assert_array_equal(lrow, lse[0, 0, rows])
        np.testing.assert_array_equal(
            oracle_mod.bwd_dq_rows(q, k, v, do, rows, causal=causal, n_valid=n_valid),
            dq[0, 0, rows])
        dkr, dvr = oracle_mod.bwd_dkdv_keys(q, k, v, do, keys, causal=causal, n_valid=n_valid)
        np.testing.assert_array_equal(dkr, dk[0, 0, keys])
        np.testing.assert_array_equal(dvr, dv[0, 0, keys])


# ---------------------------------------------------------------- value width d_v != d
# The definition puts no constraint between the key width d and the value
# width d_v: scores use d, outputs have d_v features.

def run_fwd_any(oracle, form, q, k, v, scale, causal, kv_len=None):
    if form == "direct":
        return oracle.fwd(q, k, v, scale, causal, kv_len=kv_len)
    if form == "lazy":
        return oracle.fwd_lazy(q, k, v, scale, causal, kv_len=kv_len)
    return oracle.fwd_chunked(q, k, v, scale, causal, query_chunk=2, key_chunk=3, kv_len=kv_len)


@pytest.mark.parametrize("form", FORWARD_FORMS)
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("d,d_v", [(5, 9), (8, 3)])
def test_value_width_matches_scipy_softmax(oracle_mod, form, causal, d, d_v):
    B, H, nq, nk = 2, 2, 6, 10
    q, k, v = rand((B, H, nq, d), 90), rand((B, H, nk, d), 91), rand((B, H, nk, d_v), 92)
    kv_len = [10, 7]
    o, lse = run_fwd_any(oracle_mod, form, q, k, v, 0.45, causal, kv_len)
    assert o.shape == (B, H, nq, d_v)
    for b in range(B):
        for h in range(H):
            s = _masked_scores(q[b, h], k[b, h], 0.45, kv_len[b], causal)
            np.testing.assert_allclose(o[b, h], softmax(s, axis=1) @ v[b, h], rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(lse[b, h], logsumexp(s, axis=1), rtol=1e-13)


@pytest.mark.parametrize("causal", [False, True])
def test_value_width_zero_query(oracle_mod, causal):
    B, H, nq, nk, d, d_v = 1, 2, 5, 8, 4, 7
    q, k, v = np.zeros((B, H, nq, d)), rand((B, H, nk, d), 93), rand((B, H, nk, d_v), 94)
    o, _ = oracle_mod.fwd(q, k, v, 0.3, causal)
    for i in range(nq):
        n = min(i + 1, nk) if causal else nk
        np.testing.assert_allclose(o[:, :, i], v[:, :, :n].mean(axis=2), rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("causal", [False, True])
def test_value_width_split_is_linear(oracle_mod, causal):
    # Attention is linear in v with weights independent of it: splitting the
    # value columns into two problems concatenates o and dv, leaves lse alone,
    # and adds the query and key gradients of the two halves.
    B, H, nq, nk, d, d_v = 2, 1, 7, 9, 4, 10
    q, k, v, do = (rand((B, H, nq, d), 95), rand((B, H, nk, d), 96), rand((B, H, nk, d_v), 97),
                   rand((B, H, nq, d_v), 98))
    cut = 3
    o, lse = oracle_mod.fwd(q, k, v, 0.8, causal)
    o1, l1 = oracle_mod.fwd(q, k, v[..., :cut], 0.8, causal)
    o2, l2 = oracle_mod.fwd(q, k, v[..., cut:], 0.8, causal)
    np.testing.assert_allclose(o, np.concatenate([o1, o2], axis=-1), rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(lse, l1, rtol=1e-14)
    np.testing.assert_allclose(lse, l2, rtol=1e-14)
    dq, dk, dv = oracle_mod.bwd(q, k, v, do, 0.8, causal)
    g1 = oracle_mod.bwd(q, k, v[..., :cut], do[..., :cut], 0.8, causal)
    g2 = oracle_mod.bwd(q, k, v[..., cut:], do[..., cut:], 0.8, causal)
    np.testing.assert_allclose(dq, g1[0] + g2[0], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dk, g1[1] + g2[1], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dv, np.concatenate([g1[2], g2[2]], axis=-1), rtol=1e-13, atol=1e-14)


@pytest.mark.parametrize("d,d_v", [(3, 5), (5, 2)])
def test_value_width_gradients_match_central_differences(oracle_mod, d, d_v):
    B, H, nq, nk = 1, 2, 4, 6
    q, k, v, do = (rand((B, H, nq, d), 99), rand((B, H, nk, d), 100), rand((B, H, nk, d_v), 101),
                   rand((B, H, nq, d_v), 102))

    def loss(q_, k_, v_):
        o, _ = oracle_mod.fwd(q_, k_, v_, 0.7, True, kv_len=[5])
        return float((o * do).sum())

    grads = oracle_mod.bwd(q, k, v, do, 0.7, True, kv_len=[5])
    h = 1e-6
    for which, grad in enumerate(grads):
        args = [q, k, v]
        fd = np.zeros_like(args[which])
        for idx in np.ndindex(fd.shape):
            a_p, a_m = list(args), list(args)
            a_p[which] = args[which].copy()
            a_m[which] = args[which].copy()
            a_p[which][idx] += h
            a_m[which][idx] -= h
            fd[idx] = (loss(*a_p) - loss(*a_m)) / (2 * h)
        err = np.abs(fd - grad).max() / max(np.abs(grad).max(), 1e-300)
        assert err < 1e-7, (which, err)


def test_value_width_subsets_match_full(oracle_mod):
    nq, nk, d, d_v = 13, 11, 3, 6
    q, k, v, do = (rand((nq, d), 103), rand((nk, d), 104), rand((nk, d_v), 105), rand((nq, d_v), 106))
    o, lse = oracle_mod.fwd(q[None, None], k[None, None], v[None, None], causal=True)
    dq, dk, dv = oracle_mod.bwd(q[None, None], k[None, None], v[None, None], do[None, None], causal=True)
    rows, keys = np.array([12, 0, 5]), np.array([10, 0, 4])
    orow, lrow = oracle_mod.fwd_rows(q, k, v, rows, causal=True)
    np.testing.assert_array_equal(orow, o[0, 0, rows])
    np.testing.assert_array_equal(lrow, lse[0, 0, rows])
    np.testing.assert_array_equal(oracle_mod.bwd_dq_rows(q, k, v, do, rows, causal=True), dq[0, 0, rows])
    dkr, dvr = oracle_mod.bwd_dkdv_keys(q, k, v, do, keys, causal=True)
    np.testing.assert_array_equal(dkr, dk[0, 0, keys])
    np.testing.assert_array_equal(dvr, dv[0, 0, keys])

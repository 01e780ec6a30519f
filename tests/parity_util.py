"""Shared helpers of the GPU parity tests: error metrics, input plumbing.

Metrics, for every output tensor of shape [..., rows, features]:

* rel_err(x, ref) = max |x - ref| / max |ref| over the whole tensor (the
  pass/fail metric the tolerances below are stated for; elementwise relative
  error is meaningless where outputs are near zero).
* row_err(x, ref) = max over rows of
      max_row |x - ref| / max(max_row |ref|, ROW_FLOOR * max |ref|):
  every row is held to the bar relative to its own scale, down to a floor of
  1e-3 of the tensor's largest element.  The whole-tensor metric alone barely
  looks at rows whose values are much smaller than the largest one (late rows
  of a causal output average thousands of values, so their entries are ~100x
  smaller than row 0's, which is one value vector); a kernel that wrote zeros
  there would pass it.
  For dQ and dK the row's scale also includes a quarter of the magnitude of
  the terms the row sums (gradient_row_scales): every row of dS sums to zero
  (the softmax Jacobian), so a gradient row can be an exact cancellation of
  O(1) terms -- causal row 0 of dQ is exactly 0, and so is almost every row
  of a saturated softmax -- and no floating-point evaluation of those terms
  gets within 2e-2 of a zero.  A term evaluated with relative error e
  (2^-9 for the 16-bit rounding of dS) moves the row by at most e times that
  magnitude, i.e. 2^-9 / (1/4) < 2e-2 of the scale; a row replaced by zeros
  is still caught unless it is below 1/200 of its terms' magnitude.
* per (batch, head) slice, rel_err is reported alongside.
* lse is float32 throughout the kernels (no 16-bit rounding enters it), so it
  is held elementwise to |x - ref| <= LSE_ABS + LSE_REL |ref|: 1e-4 absolute,
  widened only by the float32 rounding of the scores themselves when logits
  are large (a score of 3000 has a float32 ulp of 2.4e-4).

Bars: 1e-5 for float32 inputs, 2e-2 for 16-bit inputs with float32
accumulation, for both rel_err and row_err.
"""
import numpy as np
import torch

TOL = {"fp32": 1e-5, "bf16": 2e-2, "fp16": 2e-2}
TORCH_DT = {"fp32": torch.float32, "bf16": torch.bfloat16, "fp16": torch.float16}
ROW_FLOOR = 1e-3
LSE_ABS = 1e-4
LSE_REL = 1e-5


def rel_err(x, ref) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    denom = np.abs(ref).max()
    if denom == 0.0:
        return float(np.abs(x).max())
    return float(np.abs(x - ref).max() / denom)


TERM_SHARE = 0.25


def _row_errs(x, ref, floor: float = ROW_FLOOR, terms=None) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    x2 = x.reshape(-1, x.shape[-1])
    r2 = ref.reshape(-1, ref.shape[-1])
    top = np.abs(r2).max()
    denom = np.maximum(np.abs(r2).max(axis=1), floor * top)
    if terms is not None:
        t = np.asarray(terms, dtype=np.float64).reshape(-1)
        assert t.shape[0] == r2.shape[0], (t.shape, r2.shape)
        denom = np.maximum(denom, TERM_SHARE * t)
    with np.errstate(divide="ignore", invalid="ignore"):
        e = np.abs(x2 - r2).max(axis=1) / denom
    return np.where(denom > 0, e, np.abs(x2).max(axis=1))


def row_err(x, ref, floor: float = ROW_FLOOR, terms=None) -> float:
    """Worst row's error relative to that row's scale (last axis = features);
    `terms` (one value per row) widens the scale of rows that are sums of
    cancelling terms, see gradient_row_scales."""
    if np.size(x) == 0:
        return 0.0
    return float(_row_errs(x, ref, floor, terms).max())


def worst_row(x, ref, floor: float = ROW_FLOOR, terms=None):
    """(flat row index, its error) of the worst row, for messages."""
    e = _row_errs(x, ref, floor, terms)
    i = int(np.argmax(e))
    return i, float(e[i])


def gradient_row_scales(q, k, v, do, lse, scale, causal=False, kv_len=None):
    """Magnitude of the terms that make up each row of dQ and dK, in float64:
        cq_i = scale max_f sum_j P_ij (|dO_i|.|v_j| + |dO_i|.|o_i|) |k_jf|,
        ck_j = scale max_f sum_i P_ij (|dO_i|.|v_j| + |dO_i|.|o_i|) |q_if|,
    with P_ij = exp(scale q_i.k_j - lse_i) on visible pairs (0 elsewhere) and
    o_i = sum_j P_ij v_j: the sums of absolute values of all the products in
    dQ_i = scale sum_j P_ij (dO_i.v_j - dO_i.o_i) k_j (and dK_j alike), whose
    inner dot products dP_ij = dO_i.v_j and D_i = dO_i.o_i cancel too.
    Tolerance bookkeeping only: the reference values come from the oracle.
    Arrays [B, H, n, features]; lse [B, H, n_q] (the oracle's)."""
    q, k, v, do, lse = (np.asarray(a, dtype=np.float64) for a in (q, k, v, do, lse))
    B, H, nq, _ = q.shape
    nk = k.shape[2]
    cq = np.zeros((B, H, nq))
    ck = np.zeros((B, H, nk))
    ii = np.arange(nq)[:, None]
    jj = np.arange(nk)[None, :]
    for b in range(B):
        n_valid = nk if kv_len is None else max(0, min(int(kv_len[b]), nk))
        vis = jj < n_valid
        if causal:
            vis = vis & (jj <= ii)
        for h in range(H):
            s = scale * (q[b, h] @ k[b, h].T)
            lrow = lse[b, h][:, None]
            with np.errstate(invalid="ignore", over="ignore"):
                p = np.where(vis & np.isfinite(lrow), np.exp(np.where(vis, s, 0.0) - np.where(
                    np.isfinite(lrow), lrow, 0.0)), 0.0)
            ado = np.abs(do[b, h])
            dp_abs = ado @ np.abs(v[b, h]).T
            d_abs = (ado * np.abs(p @ v[b, h])).sum(axis=1)
            t = p * (dp_abs + d_abs[:, None])
            cq[b, h] = scale * (t @ np.abs(k[b, h])).max(axis=1)
            ck[b, h] = scale * (t.T @ np.abs(q[b, h])).max(axis=1)
    return cq, ck


def lse_err(x, ref) -> float:
    """max |x - ref| / (LSE_ABS + LSE_REL |ref|); equal infinities (a row with
    no visible key has lse = -inf on both sides) count as exact."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, (x.shape, ref.shape)
    if x.size == 0:
        return 0.0
    same_inf = np.isinf(x) & np.isinf(ref) & (np.sign(x) == np.sign(ref))
    with np.errstate(invalid="ignore"):
        d = np.where(same_inf, 0.0, np.abs(x - ref))
    scale = LSE_ABS + LSE_REL * np.where(np.isfinite(ref), np.abs(ref), 0.0)
    e = d / scale
    return float(np.nan_to_num(e, nan=np.inf, posinf=np.inf).max())


def slice_errs(x, ref, lead: int = 2):
    """rel_err of every slice over the first `lead` axes (batch, head)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    out = {}
    for idx in np.ndindex(*x.shape[:lead]):
        out[idx] = rel_err(x[idx], ref[idx])
    return out


def check(name: str, got, ref, tol: float, row_tol: float | None = None, lead: int = 2,
          terms=None) -> dict:
    """Asserts rel_err <= tol and row_err <= row_tol (default tol) for one
    output tensor, printing both and the worst (batch, head) slice; returns
    the figures.  `terms`: per-row term magnitudes for dQ and dK rows
    (gradient_row_scales), None for outputs that are not such sums."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    row_tol = tol if row_tol is None else row_tol
    assert np.all(np.isfinite(got)), (name, "non-finite values")
    e_all = rel_err(got, ref)
    e_row = row_err(got, ref, terms=terms)
    worst = ""
    if got.ndim >= lead + 2:
        se = slice_errs(got, ref, lead)
        k = max(se, key=se.get)
        worst = " worst slice %s %.3g" % (k, se[k])
    print("   %s rel_err %.3g row_err %.3g%s" % (name, e_all, e_row, worst), flush=True)
    assert e_all <= tol, (name, "rel_err", e_all, tol)
    if e_row > row_tol:
        i, e = worst_row(got, ref, terms=terms)
        raise AssertionError((name, "row_err", e_row, row_tol, "flat row", i, e))
    return {"rel": e_all, "row": e_row}


def check_lse(got, ref) -> float:
    e = lse_err(got, ref)
    print("   LSE err/(1e-4 + 1e-5|lse|) %.3g" % e, flush=True)
    assert e <= 1.0, ("LSE", e)
    return e


def f64(t: torch.Tensor) -> np.ndarray:
    """Exact widening of a (CPU or GPU) tensor to a float64 numpy array."""
    return t.detach().to("cpu", torch.float64).numpy()


def to_gpu(inputs: dict) -> dict:
    return {k: v.to("cuda") for k, v in inputs.items()}

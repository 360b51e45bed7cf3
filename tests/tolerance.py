"""Acceptance check of a binary-delta matmul result against the fp64 oracle.

Tolerance-based differential testing, as in the paper's correctness criterion
(Section 3.1, Eq. 1: outputs equal within absolute/relative tolerances, not
bitwise).  The two bars used for floating-point outputs:

  * relative Frobenius error  ||y - y_ref||_F / ||y_ref||_F  <= 5e-3
  * per element |y[m,n] - y_ref[m,n]| <= 1e-2 * ||x[m,:]||_2 * Wmax

with Wmax = max|W_base| + max_t |alpha_t| over the tenants in use: an upper
bound on the magnitude of the effective weight W_base + alpha_t * s_t.
"""
from __future__ import annotations

import numpy as np

REL_FROB = 5e-3
ELEM_FACTOR = 1e-2


def bf16_to_f64(bits):
    return (np.asarray(bits, dtype=np.uint32) << 16).view(np.float32).astype(np.float64)


def half_to_f64(bits, dtype="bf16"):
    if dtype == "f16":
        return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)
    return bf16_to_f64(bits)


def check(y, y_ref, x_bits, w_bits, alpha, tenant_ids=None, rows=None,
          rel_frob=REL_FROB, elem_factor=ELEM_FACTOR, dtype="bf16"):
    """Raise AssertionError with a diagnostic when y misses either bar.

    y, y_ref: float arrays [M', C] (C sampled columns); rows: the x rows they
    belong to (default all).  Returns (relF, worst element ratio).
    """
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    assert y.shape == y_ref.shape, (y.shape, y_ref.shape)
    assert np.all(np.isfinite(y_ref)), "reference has non-finite entries"
    assert np.all(np.isfinite(y)), f"result has {np.count_nonzero(~np.isfinite(y))} non-finite entries"
    x = half_to_f64(x_bits, dtype)
    if rows is not None:
        x = x[np.asarray(rows)]
    alpha = np.atleast_1d(np.asarray(alpha, dtype=np.float64))
    used = alpha if tenant_ids is None else alpha[np.unique(np.asarray(tenant_ids))]
    wmax = float(np.max(np.abs(half_to_f64(w_bits, dtype)))) + float(np.max(np.abs(used)))
    num = np.linalg.norm(y - y_ref)
    den = np.linalg.norm(y_ref)
    relf = num / den if den > 0 else num
    bound = elem_factor * np.linalg.norm(x, axis=1)[:, None] * wmax
    err = np.abs(y - y_ref)
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(bound > 0, err / bound, np.where(err > 0, np.inf, 0.0))
    worst = float(np.max(ratio)) if ratio.size else 0.0
    assert relf <= rel_frob, f"relative Frobenius error {relf:.3e} > {rel_frob:.1e}"
    assert worst <= 1.0, f"per-element error reaches {worst:.3f} of its bound"
    return relf, worst

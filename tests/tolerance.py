"""Comparison rules between the GPU library and the oracle.

Integers (ids, counts, offsets, owners): bit-exact.

Coalesced gradient sums: element-wise |gpu - exact| <= rtol * sum|g|, where
`exact` is the oracle's fp64 sum and sum|g| its sum of magnitudes.  This is
the scale of the standard error bound of a floating-point sum (Higham,
Accuracy and Stability of Numerical Algorithms, Sec. 4.2): any summation
order in fp32 over n terms errs by at most about (n-1) * 2^-24 * sum|g|, so a
plain relative error would wrongly fail sums that cancel.  rtol = 1e-5 for
fp32 gradients; the bf16-gradient bar is 2e-2 (the same metric is reported
for it too).

Rows of W, m, v after an update: row-wise max-norm,
||gpu_row - orc_row||_inf <= rtol * ||orc_row||_inf.

The update itself, dW = W_after - W_before: the check above measures a W row
against its own size (about 3 for N(0, 1) weights), about 3e-5 per element,
which would let through an error of a few percent of an update of about lr =
1e-3.  So the change is judged on its own scale, element by element:
|W_gpu - W_orc| <= rtol * ||dW_orc_row||_inf + k * ulp(W_orc), where the first
term bounds the error of the fp32 update arithmetic (a handful of roundings,
far below rtol relative to the update) and the second the final rounding of
w - update to fp32, which both sides do (up to one unit in the last place per
update; k updates in a chain).  Kingma & Ba, Algorithm 1: the update is
lr * m_hat / (sqrt(v_hat) + eps); where |g| is near eps / sqrt(1 - b2^t) a
misplaced eps changes it by up to ~lr, far beyond this bound.
"""
from __future__ import annotations

import numpy as np

RTOL_F32 = 1e-5
RTOL_BF16 = 2e-2


def grad_error_ratio(gpu, exact_f64, absum):
    """max over elements of |gpu - exact| / sum|g| (0/0 counts as 0; x/0 as inf)."""
    gpu = np.asarray(gpu, dtype=np.float64)
    err = np.abs(gpu - exact_f64)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(absum > 0, err / np.where(absum > 0, absum, 1.0), np.where(err > 0, np.inf, 0.0))
    return float(r.max()) if r.size else 0.0


def assert_grad_close(gpu, exact_f64, absum, rtol=RTOL_F32, what="coalesced gradient"):
    r = grad_error_ratio(gpu, exact_f64, absum)
    assert r <= rtol, f"{what}: max |gpu-exact|/sum|g| = {r:.3e} > {rtol:.1e}"
    return r


def row_error_ratio(gpu, ref):
    """max over rows of ||gpu - ref||_inf / ||ref||_inf."""
    gpu = np.asarray(gpu, dtype=np.float64).reshape(len(ref), -1) if len(ref) else np.zeros((0, 1))
    ref = np.asarray(ref, dtype=np.float64).reshape(len(ref), -1) if len(ref) else np.zeros((0, 1))
    if ref.size == 0:
        return 0.0
    num = np.abs(gpu - ref).max(axis=1)
    den = np.abs(ref).max(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(den > 0, num / np.where(den > 0, den, 1.0), np.where(num > 0, np.inf, 0.0))
    return float(r.max())


def assert_rows_close(gpu, ref, rtol=RTOL_F32, what="rows"):
    r = row_error_ratio(gpu, ref)
    assert r <= rtol, f"{what}: max row ||gpu-ref||_inf/||ref||_inf = {r:.3e} > {rtol:.1e}"
    return r


def update_error_ratio(gpu, before, ref, ulps=1):
    """max over elements of max(|gpu - ref| - ulps * ulp(ref), 0) / ||ref_row - before_row||_inf
    (0/0 counts as 0, x/0 as inf): the error of the update beyond the final roundings, relative to
    the row's update."""
    n = len(ref)
    if n == 0:
        return 0.0
    gpu = np.asarray(gpu, dtype=np.float64).reshape(n, -1)
    before = np.asarray(before, dtype=np.float64).reshape(n, -1)
    ref32 = np.asarray(ref, dtype=np.float32).reshape(n, -1)
    ref = ref32.astype(np.float64)
    ulp = np.spacing(np.abs(ref32)).astype(np.float64)
    excess = np.maximum(np.abs(gpu - ref) - ulps * ulp, 0.0)
    scale = np.abs(ref - before).max(axis=1, keepdims=True)
    with np.errstate(divide="ignore", invalid="ignore"):
        r = np.where(scale > 0, excess / np.where(scale > 0, scale, 1.0), np.where(excess > 0, np.inf, 0.0))
    return float(r.max())


def assert_update_close(gpu, before, ref, rtol=RTOL_F32, ulps=1, what="update"):
    r = update_error_ratio(gpu, before, ref, ulps)
    assert r <= rtol, f"{what}: max (|gpu-ref| - {ulps} ulp)/||dW_row||_inf = {r:.3e} > {rtol:.1e}"
    return r

"""The update tolerance (tests/tolerance.py) must tell a correct fp32 evaluation of Kingma & Ba's
Algorithm 1 (Sec. 5.7 of the paper: Adam with one step counter per iteration) from plausible
mistakes in the final W formula, with gradients that include the regime where eps matters (|g| near
eps / sqrt(1 - b2^t)) and zeros: the placement of eps, and a step size off by a fraction of a
percent, which the older row check (W rows against their own max-norm) lets through.  CPU only: a float32 evaluation written here in numpy stands in for
the kernel's arithmetic; the reference is the oracle."""
import numpy as np
import pytest

import oracle
import tolerance
from adam_inputs import eps_regime_grads

LR, B1, B2, EPS = 1e-3, 0.9, 0.999, 1e-8


def adam_f32(W, m, v, g, step, form="alg1", lr_scale=1.0):
    """Algorithm 1 evaluated in float32 as the kernel does: fp64 bias corrections turned into fp32
    coefficients, then m, v, w per element.  form="pytorch": PyTorch's SparseAdam ordering
    (lr sqrt(bc2) / bc1 * m / (sqrt(v) + eps)), i.e. eps effectively divided by sqrt(bc2)."""
    f = np.float32
    bc1 = 1.0 - B1 ** step
    bc2 = 1.0 - B2 ** step
    m = f(B1) * m + f(1.0 - B1) * g
    v = f(B2) * v + f(1.0 - B2) * (g * g)
    if form == "alg1":
        upd = f(LR * lr_scale / bc1) * (m / (np.sqrt(v * f(1.0 / bc2)) + f(EPS)))
    else:
        upd = f(LR * lr_scale * np.sqrt(bc2) / bc1) * (m / (np.sqrt(v) + f(EPS)))
    return (W - upd).astype(np.float32), m.astype(np.float32), v.astype(np.float32)


def run(form, steps=3, lr_scale=1.0, seed=5):
    rng = np.random.default_rng(seed)
    n, D = 64, 32
    W = rng.normal(0.0, 1.0, (n, D)).astype(np.float32)
    m = np.zeros_like(W)
    v = np.zeros_like(W)
    worst_upd, worst_row = 0.0, 0.0
    for t in range(1, steps + 1):
        g = eps_regime_grads(rng, n, D)
        Wr, mr, vr = W.copy(), m.copy(), v.copy()
        oracle.sparse_adam(Wr, mr, vr, np.arange(n, dtype=np.int32), g, np.array([0, n], np.int32), 0, 1,
                           LR, B1, B2, EPS, t)
        Wg, mg, vg = adam_f32(W, m, v, g, t, form, lr_scale)
        worst_upd = max(worst_upd, tolerance.update_error_ratio(Wg, W, Wr))
        worst_row = max(worst_row, tolerance.row_error_ratio(Wg, Wr))
        W, m, v = Wr, mr, vr  # each call judged on identical inputs: continue from the oracle's state
    return worst_upd, worst_row


def test_correct_fp32_update_passes():
    upd, row = run("alg1")
    assert upd <= tolerance.RTOL_F32 and row <= tolerance.RTOL_F32, (upd, row)


def test_eps_placement_is_caught_in_the_eps_regime():
    upd, _ = run("pytorch")
    assert upd > 100 * tolerance.RTOL_F32, upd


@pytest.mark.parametrize("scale", [1.01, 0.999])
def test_small_step_size_error_is_caught_by_the_update_check_only(scale):
    upd, row = run("alg1", lr_scale=scale)
    assert upd > 10 * tolerance.RTOL_F32, upd
    assert row <= tolerance.RTOL_F32, row


def test_untouched_elements_and_zero_rows():
    # a zero gradient on fresh moments leaves w exactly as it was: no update, no allowance beyond rounding
    W = np.array([[1.0, -2.0, 0.5]], np.float32)
    assert tolerance.update_error_ratio(W, W, W) == 0.0
    assert tolerance.update_error_ratio(W + np.float32(1e-3), W, W) == np.inf

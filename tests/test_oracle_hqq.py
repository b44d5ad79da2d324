"""Pins of the HQQ-style zero-point oracle (oracle/hqq.py): the zero step against a
library least-squares solve, the threshold operator against its closed forms (the
soft threshold at p = 1, the identity as beta grows, a hand value), weights on an
exact grid (min/max is already perfect and must be kept), the never-worse invariant,
a measurable gain over min/max on Gaussian weights (a dropped threshold, a wrong
sign in the zero step or a broken stopping rule all remove it), degenerate groups,
and a pure-Python run of the rounds on one small group."""
import math

import numpy as np
import pytest

import oracle
from oracle.hqq import (HQQ_BETA, HQQ_ITERS, HQQ_KAPPA, HQQ_P, group_l1, optimise_zero, quantize_hqq,
                        shrink_lp, zero_step)


def test_zero_step_is_the_least_squares_fit():
    rng = np.random.default_rng(0)
    w = rng.normal(0, 0.02, (5, 64))
    s = np.full(5, 0.004)
    q = np.clip(np.rint(w / s[:, None] + 7.3), 0, 15)
    e = rng.normal(0, 0.001, (5, 64))
    z = zero_step(w, q, e, s)
    for g in range(5):
        # minimise || (q - (w - e)/s) - z * 1 ||^2 over the scalar z
        sol, *_ = np.linalg.lstsq(np.ones((64, 1)), q[g] - (w[g] - e[g]) / s[g], rcond=None)
        assert math.isclose(z[g], sol[0], rel_tol=0, abs_tol=1e-12)


def test_threshold_operator_closed_forms():
    x = np.array([-3.0, -0.5, -0.1, 0.0, 0.05, 0.4, 2.0])
    # p = 1: the soft threshold by 1/beta
    assert np.allclose(shrink_lp(x, 4.0, 1.0), np.sign(x) * np.maximum(np.abs(x) - 0.25, 0.0), atol=0, rtol=0)
    # a very large beta leaves x unchanged (to rounding)
    assert np.allclose(shrink_lp(x, 1e30, HQQ_P), x, atol=1e-15)
    # hand value: x = 2, p = 0.5, beta = 1: 2 - 2^-0.5
    assert math.isclose(shrink_lp(np.array([2.0]), 1.0, 0.5)[0], 2.0 - 2.0 ** -0.5, abs_tol=1e-15)
    # small magnitudes are set to zero (|x|^(p-1) / beta exceeds |x|), zero stays zero
    assert shrink_lp(np.array([1e-4, 0.0, -1e-4]), HQQ_BETA, HQQ_P).tolist() == [0.0, 0.0, 0.0]


def test_weights_on_an_exact_grid_keep_the_min_max_result():
    s, z0 = 2.0 ** -6, 7.0
    rng = np.random.default_rng(1)
    q = rng.integers(0, 16, (8, 128)).astype(np.float64)
    q[:, 0], q[:, 1] = 0, 15  # every group of 64 spans the full range
    q[:, 64], q[:, 65] = 0, 15
    w = ((q - z0) * s).astype(np.float32)
    qh, sh, zh = quantize_hqq(w, 4, 64)
    q0, s0, z00 = oracle.quantize_minmax(w, 4, 64)
    assert np.array_equal(qh, q0) and np.array_equal(sh, s0) and np.array_equal(zh, z00)
    assert np.array_equal(qh, q.astype(np.uint8))
    assert np.all(zh == np.float16(z0))


@pytest.mark.parametrize("bits,group", [(4, 64), (3, 64), (2, 64), (4, 128)])
def test_never_worse_and_better_on_average(bits, group):
    rng = np.random.default_rng(bits * 10 + group)
    w = (rng.standard_normal((64, 1024)) * 0.02).astype(np.float32)
    qh, sh, zh = quantize_hqq(w, bits, group)
    q0, s0, z0 = oracle.quantize_minmax(w, bits, group)
    assert np.array_equal(sh, s0)  # the scale is not touched
    qmax = float(2 ** bits - 1)
    wg = w.astype(np.float64).reshape(64, 1024 // group, group)
    eh = group_l1(wg, sh.T.astype(np.float64), zh.T.astype(np.float64), qmax)
    e0 = group_l1(wg, s0.T.astype(np.float64), z0.T.astype(np.float64), qmax)
    assert np.all(eh <= e0)
    assert eh.sum() < 0.985 * e0.sum()
    # the codes are the rounding rule applied with the returned scale and zero
    t = np.clip(np.rint(wg / sh.T.astype(np.float64)[:, :, None] + zh.T.astype(np.float64)[:, :, None]), 0, qmax)
    assert np.array_equal(qh, t.reshape(64, 1024).astype(np.uint8))


def test_degenerate_groups_match_min_max():
    w = np.zeros((4, 128), np.float32)
    w[1, :64] = 0.25
    w[2, 64:] = np.linspace(-1, 1, 64, dtype=np.float32)
    qh, sh, zh = quantize_hqq(w, 4, 64)
    q0, s0, z0 = oracle.quantize_minmax(w, 4, 64)
    assert np.array_equal(sh, s0)
    const = np.ones((4, 2), bool)
    const[2, 1] = False  # the one group with a spread
    assert np.array_equal(zh.T[const], z0.T[const]) and np.array_equal(qh.reshape(4, 2, 64)[const],
                                                                         q0.reshape(4, 2, 64)[const])


def test_rounds_match_a_plain_python_run():
    rng = np.random.default_rng(3)
    w = [float(v) for v in rng.normal(0, 0.02, 16)]
    qmax = 3.0
    wmin, wmax = min(w), max(w)
    s = float(np.float16((wmax - wmin) / qmax))
    z0 = float(np.float16(-wmin / s))

    def l1(z):
        tot = 0.0
        for v in w:
            q = min(max(round_half_even(v / s + z), 0.0), qmax)
            tot += abs(v - (q - z) * s)
        return tot

    def round_half_even(t):
        return float(np.rint(t))

    z, best_z, best = z0, z0, l1(z0)
    beta = HQQ_BETA
    for _ in range(HQQ_ITERS):
        acc = 0.0
        for v in w:
            q = min(max(round_half_even(v / s + z), 0.0), qmax)
            x = v - (q - z) * s
            e = math.copysign(max(abs(x) - abs(x) ** (HQQ_P - 1) / beta, 0.0), x) if x != 0 else 0.0
            acc += q - (v - e) / s
        z_new = acc / len(w)
        err = l1(z_new)
        if not err < best:
            break
        best, best_z, z = err, z_new, z_new
        beta *= HQQ_KAPPA
    bz, be = optimise_zero(np.array([w]), np.array([s]), np.array([z0]), qmax)
    assert math.isclose(bz[0], best_z, rel_tol=0, abs_tol=1e-12) and math.isclose(be[0], best, abs_tol=1e-12)

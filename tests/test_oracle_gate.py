"""Pins of the fp64 output-gate reference (the mixer's last line in Alg. 2:
RMSNorm of the head's output times a sigmoid gate) against values fixed by
the definition, not by re-typing the oracle's formulas."""
import math

import numpy as np

import oracle


def test_worked_example():
    # o = (3, 4): mean square 12.5, so o / rms = (3, 4) * sqrt(2) / 5; gain
    # (1, 2); gates sigmoid(0) = 1/2 and sigmoid(ln 3) = 3/4 (eps = 0):
    # y = (3 sqrt(2) / 10, 6 sqrt(2) / 5)
    y = oracle.out_gate_fwd([[3.0, 4.0]], [[0.0, math.log(3.0)]], [1.0, 2.0], 0.0)
    np.testing.assert_allclose(y[0], [3 * math.sqrt(2) / 10, 6 * math.sqrt(2) / 5], rtol=1e-15)


def test_unit_rms_with_open_gate():
    rng = np.random.default_rng(1)
    o = rng.standard_normal((5, 3, 16))
    y = oracle.out_gate_fwd(o, np.full_like(o, 60.0), np.ones(16), 0.0)
    np.testing.assert_allclose(np.mean(y * y, axis=-1), 1.0, rtol=1e-12)


def test_scale_invariance_and_zero_row():
    rng = np.random.default_rng(2)
    o = rng.standard_normal((4, 32))
    z = rng.standard_normal((4, 32))
    w = rng.standard_normal(32)
    np.testing.assert_allclose(oracle.out_gate_fwd(7.5 * o, z, w, 0.0), oracle.out_gate_fwd(o, z, w, 0.0),
                               rtol=1e-13)
    o[1] = 0.0
    y = oracle.out_gate_fwd(o, z, w, 1e-6)
    assert np.all(np.isfinite(y)) and np.all(y[1] == 0.0)


def test_gradients_match_finite_differences():
    rng = np.random.default_rng(3)
    shape, V, eps = (3, 2, 8), 8, 1e-3
    o = rng.standard_normal(shape)
    z = rng.standard_normal(shape)
    w = rng.standard_normal(V)
    dy = rng.standard_normal(shape)
    do, dz, dw = oracle.out_gate_bwd(o, z, w, eps, dy)

    def loss(o_, z_, w_):
        return float(np.sum(dy * oracle.out_gate_fwd(o_, z_, w_, eps)))
    h = 1e-6
    for name, x, g in (("o", o, do), ("z", z, dz), ("w", w, dw)):
        fd = np.zeros_like(x)
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args = {"o": o, "z": z, "w": w}
            args[name] = xp
            lp = loss(args["o"], args["z"], args["w"])
            args[name] = xm
            lm = loss(args["o"], args["z"], args["w"])
            fd[idx] = (lp - lm) / (2 * h)
        np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-8, err_msg=name)


def test_gain_gradient_adds_over_rows():
    rng = np.random.default_rng(4)
    o = rng.standard_normal((6, 16))
    z = rng.standard_normal((6, 16))
    w = rng.standard_normal(16)
    dy = rng.standard_normal((6, 16))
    do1, dz1, dw1 = oracle.out_gate_bwd(o, z, w, 1e-6, dy)
    do2, dz2, dw2 = oracle.out_gate_bwd(np.concatenate([o, o]), np.concatenate([z, z]), w, 1e-6,
                                        np.concatenate([dy, dy]))
    np.testing.assert_allclose(dw2, 2 * dw1, rtol=1e-14)
    np.testing.assert_allclose(do2[:6], do1, rtol=0, atol=0)
    np.testing.assert_allclose(dz2[6:], dz1, rtol=0, atol=0)

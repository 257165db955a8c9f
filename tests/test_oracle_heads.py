"""Pins of the fp64 gate-head reference (Alg. 2: alpha = exp(-exp(A)
softplus(x + b)), beta = sigmoid(x_beta)) against values the definition
fixes, and its backward against finite differences."""
import math

import numpy as np

import oracle


def test_worked_example():
    # A = 0, b = 0, x = 0: softplus(0) = ln 2, so g = -ln 2 and alpha = 1/2;
    # A = ln 3, x + b = ln(e - 1): softplus = 1, g = -3; sigmoid(0) = 1/2
    g, beta = oracle.gate_heads_fwd([[[0.0, math.log(math.e - 1.0) - 0.5]]], [[0.0]],
                                    [[0.0, math.log(3.0)]], [[0.0, 0.5]])
    np.testing.assert_allclose(g[0, 0], [-math.log(2.0), -3.0], rtol=1e-14)
    np.testing.assert_allclose(beta[0, 0], 0.5, rtol=0)


def test_gate_is_a_decay_and_limits():
    rng = np.random.default_rng(1)
    x = 30.0 * rng.standard_normal((50, 2, 4))
    A = rng.standard_normal((2, 4))
    b = rng.standard_normal((2, 4))
    g, _ = oracle.gate_heads_fwd(x, np.zeros((50, 2)), A, b)
    assert np.all(g <= 0.0) and np.all(np.isfinite(g))
    # x + b -> -inf: softplus -> 0, no decay; x + b -> +inf: g -> -exp(A)(x + b)
    g0, _ = oracle.gate_heads_fwd(np.full((1, 2, 4), -800.0), np.zeros((1, 2)), A, b)
    np.testing.assert_allclose(g0, 0.0, atol=1e-300)
    xl = np.full((1, 2, 4), 700.0)
    gl, _ = oracle.gate_heads_fwd(xl, np.zeros((1, 2)), A, b)
    np.testing.assert_allclose(gl, -np.exp(A) * (xl + b), rtol=1e-12)


def test_gradients_match_finite_differences():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 2, 4))
    xb = rng.standard_normal((3, 2))
    A = 0.5 * rng.standard_normal((2, 4))
    b = rng.standard_normal((2, 4))
    dg = rng.standard_normal((3, 2, 4))
    dbeta = rng.standard_normal((3, 2))
    grads = dict(zip(("x", "xb", "A", "b"), oracle.gate_heads_bwd(x, xb, A, b, dg, dbeta)))
    args = {"x": x, "xb": xb, "A": A, "b": b}

    def loss(a):
        g, beta = oracle.gate_heads_fwd(a["x"], a["xb"], a["A"], a["b"])
        return float(np.sum(dg * g) + np.sum(dbeta * beta))
    h = 1e-6
    for name in args:
        fd = np.zeros_like(args[name])
        for idx in np.ndindex(fd.shape):
            ap = {k: v.copy() for k, v in args.items()}
            am = {k: v.copy() for k, v in args.items()}
            ap[name][idx] += h
            am[name][idx] -= h
            fd[idx] = (loss(ap) - loss(am)) / (2 * h)
        np.testing.assert_allclose(grads[name], fd, rtol=1e-6, atol=1e-9, err_msg=name)


def test_write_strength_slope_in_the_tails():
    """d sigmoid / dx = e^-|x| / (1 + e^-|x|)^2 exactly; in the tails this is
    tiny but still owed to full relative precision (1 - sigmoid(x) would round
    to 0 in fp64 beyond |x| ~ 37)."""
    xb = np.array([[-60.0, -40.0, -5.0, 0.0, 5.0, 40.0, 60.0]])
    _, dxb, _, _ = oracle.gate_heads_bwd(np.zeros((1, 7, 1)), xb, np.zeros((7, 1)), np.zeros((7, 1)),
                                         np.zeros((1, 7, 1)), np.ones((1, 7)))
    a = np.exp(-np.abs(xb))
    np.testing.assert_allclose(dxb, a / (1.0 + a) ** 2, rtol=1e-13, atol=0)


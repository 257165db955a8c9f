"""Pins of the fp64 input-side reference (causal depthwise convolution, SiLU
on q, k, v, softplus on q', k', L2 normalisation of q, k, q', k'; section
"Input projections" and Alg. 2) against a hand-worked example, numpy's own
convolution, causality, unit norms, and its backward against central finite
differences."""
import math

import numpy as np

import oracle.conv_in as ci


def test_worked_example():
    """H = 1, K = 2, V = 1, E = 2, W = 2 with taps (0.5, 1) on every channel,
    eps = 0.  Token 0 sees only itself; token 1 sees 0.5 y[0] + y[1].
      q: y0 = (ln 3, -ln 3), y1 = (ln 3, -ln 3) / 2  ->  z = (ln 3, -ln 3) at
         both tokens; SiLU = ln 3 (3/4, -1/4); normalised (3, -1) / sqrt 10.
      k: y0 = (-ln 3, ln 3)  ->  token 0: (-1, 3) / sqrt 10 (token 1 is
         not checked: SiLU is not homogeneous, so z = y0 / 2 changes the
         direction).
      v: y0 = ln 3, y1 = 0  ->  v0 = (3/4) ln 3; z1 = (ln 3) / 2,
         sigmoid((ln 3)/2) = sqrt 3 / (1 + sqrt 3), v1 = z1 times that.
      q': y0 = (ln(e - 1), ln(e - 1)) -> softplus (1, 1) -> (1, 1) / sqrt 2.
      k': y0 = (0, ln(e - 1)) -> (ln 2, 1) / sqrt(ln^2 2 + 1)."""
    l3, le = math.log(3.0), math.log(math.e - 1.0)
    y = np.zeros((1, 2, 2 * 2 + 1 + 2 * 2))
    y[0, 0] = [l3, -l3, -l3, l3, l3, le, le, 0.0, le]
    y[0, 1] = [l3 / 2, -l3 / 2, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0]
    w = np.stack([np.full(9, 0.5), np.ones(9)])
    o = ci.conv_in_fwd(y, w, 1, 2, 1, 2, 0.0)
    s10 = math.sqrt(10.0)
    np.testing.assert_allclose(o["q"][0, 0, 0], [3 / s10, -1 / s10], rtol=1e-14)
    np.testing.assert_allclose(o["q"][0, 1, 0], [3 / s10, -1 / s10], rtol=1e-14)
    np.testing.assert_allclose(o["k"][0, 0, 0], [-1 / s10, 3 / s10], rtol=1e-14)
    np.testing.assert_allclose(o["v"][0, 0, 0], [0.75 * l3], rtol=1e-14)
    r3 = math.sqrt(3.0)
    np.testing.assert_allclose(o["v"][0, 1, 0], [l3 / 2 * r3 / (1 + r3)], rtol=1e-14)
    np.testing.assert_allclose(o["q2"][0, 0, 0], [1 / math.sqrt(2.0)] * 2, rtol=1e-14)
    n = math.sqrt(math.log(2.0) ** 2 + 1.0)
    np.testing.assert_allclose(o["k2"][0, 0, 0], [math.log(2.0) / n, 1 / n], rtol=1e-14)


def test_convolution_is_numpys_causal_convolution():
    rng = np.random.default_rng(3)
    for W in (1, 2, 3, 4):
        y = rng.standard_normal((2, 11, 5))
        w = rng.standard_normal((W, 5))
        z = ci.causal_conv(y, w)
        for b in range(2):
            for c in range(5):
                ref = np.convolve(y[b, :, c], w[::-1, c])[:11]
                np.testing.assert_allclose(z[b, :, c], ref, rtol=1e-13, atol=1e-13)


def test_causal_and_rows_independent():
    rng = np.random.default_rng(4)
    H, K, V, E, W = 2, 4, 3, 2, 3
    C = H * (2 * K + V + 2 * E)
    y = rng.standard_normal((2, 9, C))
    w = rng.standard_normal((W, C))
    base = ci.conv_in_fwd(y, w, H, K, V, E, 1e-6)
    y2 = y.copy()
    y2[1, 4] += 1.0  # token 4 of row 1
    pert = ci.conv_in_fwd(y2, w, H, K, V, E, 1e-6)
    for name in base:
        d = np.abs(pert[name] - base[name]).reshape(2, 9, -1).max(axis=-1)
        assert np.all(d[0] == 0), name           # other batch row untouched
        assert np.all(d[1, :4] == 0), name        # earlier tokens untouched
        assert np.all(d[1, 4 + W:] == 0), name    # beyond the window untouched
        assert np.all(d[1, 4:4 + W] > 0), name


def test_unit_norms_and_unnormalised_values():
    rng = np.random.default_rng(5)
    H, K, V, E, W = 3, 8, 5, 4, 4
    C = H * (2 * K + V + 2 * E)
    y = rng.standard_normal((2, 7, C))
    w = rng.standard_normal((W, C))
    o = ci.conv_in_fwd(y, w, H, K, V, E, 0.0)
    for name in ("q", "k", "q2", "k2"):
        np.testing.assert_allclose(np.linalg.norm(o[name], axis=-1), 1.0, rtol=1e-13)
    assert np.all(o["q2"] > 0) and np.all(o["k2"] > 0)  # softplus channels stay positive
    z = ci.causal_conv(y, w)[:, :, 2 * H * K:2 * H * K + H * V]
    np.testing.assert_allclose(o["v"].reshape(2, 7, -1), z / (1.0 + np.exp(-z)), rtol=1e-13)


def test_gradients_match_finite_differences():
    rng = np.random.default_rng(6)
    H, K, V, E, W, eps = 2, 3, 2, 2, 3, 1e-3
    C = H * (2 * K + V + 2 * E)
    y = rng.standard_normal((2, 5, C))
    w = rng.standard_normal((W, C))
    shapes = {"q": K, "k": K, "v": V, "q2": E, "k2": E}
    grads = {n: rng.standard_normal((2, 5, H, d)) for n, d in shapes.items()}

    def loss(y_, w_):
        o = ci.conv_in_fwd(y_, w_, H, K, V, E, eps)
        return sum(np.sum(grads[n] * o[n]) for n in shapes)

    dy, dw = ci.conv_in_bwd(y, w, H, K, V, E, eps, grads)
    h = 1e-6
    num = np.zeros_like(y)
    for i in np.ndindex(y.shape):
        yp, ym = y.copy(), y.copy()
        yp[i] += h
        ym[i] -= h
        num[i] = (loss(yp, w) - loss(ym, w)) / (2 * h)
    np.testing.assert_allclose(dy, num, rtol=1e-6, atol=1e-8)
    numw = np.zeros_like(w)
    for i in np.ndindex(w.shape):
        wp, wm = w.copy(), w.copy()
        wp[i] += h
        wm[i] -= h
        numw[i] = (loss(y, wp) - loss(y, wm)) / (2 * h)
    np.testing.assert_allclose(dw, numw, rtol=1e-6, atol=1e-8)

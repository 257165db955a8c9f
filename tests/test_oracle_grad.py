"""Pins of the oracle's reverse-mode backward: central finite differences of
the forward, entry by entry on a tiny problem, and a directional (adjoint) check
on a larger one.  The loss is L = <o, dO> + <s_final, dS_final>."""
import numpy as np
import pytest

import oracle

SGLA, GDN = oracle.SGLA, oracle.GDN
NAMES = ["q", "k", "v", "q2", "k2", "g", "beta", "s0"]
GRAD = {"q": "dq", "k": "dk", "v": "dv", "q2": "dq2", "k2": "dk2", "g": "dg",
        "beta": "dbeta", "s0": "ds0"}


def make(rng, B, T, H, K, V, E, with_beta=True):
    def unit(shape):
        x = rng.standard_normal(shape)
        return x / np.linalg.norm(x, axis=-1, keepdims=True)
    d = dict(q=unit((B, T, H, K)), k=unit((B, T, H, K)), v=rng.standard_normal((B, T, H, V)),
             q2=unit((B, T, H, E)), k2=unit((B, T, H, E)),
             g=rng.uniform(-0.6, -0.01, (B, T, H, E)),
             beta=rng.uniform(0.1, 0.95, (B, T, H)) if with_beta else None,
             s0=0.5 * rng.standard_normal((B, H, E, K, V)))
    dO = rng.standard_normal((B, T, H, V))
    dSf = rng.standard_normal((B, H, E, K, V))
    return d, dO, dSf


def loss(variant, d, dO, dSf):
    o, sf = oracle.fwd(variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], d["s0"])
    return float(np.sum(o * dO) + np.sum(sf * dSf))


@pytest.mark.parametrize("variant,with_beta", [(GDN, True), (SGLA, True), (SGLA, False)])
def test_finite_differences_every_entry(variant, with_beta):
    rng = np.random.default_rng(20 + variant + 2 * with_beta)
    d, dO, dSf = make(rng, B=1, T=11, H=2, K=3, V=2, E=2, with_beta=with_beta)
    gr = oracle.bwd(variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"],
                    d["s0"], dO, dSf)
    h = 1e-6
    for name in NAMES:
        if d[name] is None:
            assert gr["dbeta"] is None
            continue
        x = d[name]
        num = np.zeros_like(x)
        for i in np.ndindex(x.shape):
            old = x[i]
            x[i] = old + h
            lp = loss(variant, d, dO, dSf)
            x[i] = old - h
            lm = loss(variant, d, dO, dSf)
            x[i] = old
            num[i] = (lp - lm) / (2 * h)
        ana = gr[GRAD[name]]
        scale = max(1.0, np.max(np.abs(num)))
        np.testing.assert_allclose(ana, num, rtol=0, atol=2e-7 * scale, err_msg=name)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_adjoint_directional(variant):
    """<grad L, delta> equals the directional derivative of L along delta."""
    rng = np.random.default_rng(30 + variant)
    d, dO, dSf = make(rng, B=2, T=70, H=2, K=6, V=5, E=3)   # crosses the 64-token segment
    gr = oracle.bwd(variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"],
                    d["s0"], dO, dSf)
    delta = {n: rng.standard_normal(d[n].shape) for n in NAMES}
    ana = sum(float(np.sum(gr[GRAD[n]] * delta[n])) for n in NAMES)
    h = 1e-5
    dp = {n: d[n] + h * delta[n] for n in NAMES}
    dm = {n: d[n] - h * delta[n] for n in NAMES}
    num = (loss(variant, dp, dO, dSf) - loss(variant, dm, dO, dSf)) / (2 * h)
    assert abs(ana - num) <= 1e-7 * max(1.0, abs(num)), (ana, num)


def test_zero_upstream_gives_zero_gradients():
    rng = np.random.default_rng(40)
    d, dO, dSf = make(rng, B=1, T=5, H=1, K=3, V=2, E=2)
    gr = oracle.bwd(GDN, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"],
                    d["s0"], np.zeros_like(dO), None)
    for key, val in gr.items():
        assert np.all(val == 0.0), key

"""Pins of the fp64 oracle against what the paper and the mathematics fix.

None of these re-types the oracle's own loop: each compares it with an
independent statement of the operator (flattened joint key, dyadic special
case, quadratic form, chunkwise form), a closed form, an invariant, or a
hand-derived worked example.
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import forms

SGLA, GDN = oracle.SGLA, oracle.GDN
HERE = os.path.dirname(os.path.abspath(__file__))


def rand_inputs(rng, B=2, T=13, H=2, K=4, V=3, E=3, with_beta=True, with_s0=True,
                gate_lo=-0.7):
    def unit(shape):
        x = rng.standard_normal(shape)
        return x / np.linalg.norm(x, axis=-1, keepdims=True)
    return dict(
        q=unit((B, T, H, K)), k=unit((B, T, H, K)), v=rng.standard_normal((B, T, H, V)),
        q2=unit((B, T, H, E)), k2=unit((B, T, H, E)),
        g=rng.uniform(gate_lo, 0.0, (B, T, H, E)),
        beta=rng.uniform(0.05, 1.0, (B, T, H)) if with_beta else None,
        s0=0.3 * rng.standard_normal((B, H, E, K, V)) if with_s0 else None,
    )


def run(variant, d):
    return oracle.fwd(variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], d["s0"])


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("with_beta", [True, False])
def test_flattened_joint_key(variant, with_beta):
    """Eq. gdn3flat: GDN (or gated LA) on the d*E joint key with per-slice decay."""
    if variant == GDN and not with_beta:
        pytest.skip("GDN always has a write strength")
    d = rand_inputs(np.random.default_rng(1), with_beta=with_beta)
    o, sf = run(variant, d)
    o2, sf2 = forms.flat_joint_key(variant, **d)
    np.testing.assert_allclose(o, o2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(sf, sf2, rtol=0, atol=1e-12)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_dyadic_reduction_E1(variant):
    """E = 1 with k' = q' = 1 is ordinary gated DeltaNet / gated LA (Eq. la3 remark,
    Appendix A remark)."""
    rng = np.random.default_rng(2)
    d = rand_inputs(rng, E=1)
    d["q2"] = np.ones_like(d["q2"])
    d["k2"] = np.ones_like(d["k2"])
    o, sf = run(variant, d)
    o2, sf2 = forms.dyadic(variant, d["q"], d["k"], d["v"], d["g"][..., 0], d["beta"],
                           d["s0"][:, :, 0])
    np.testing.assert_allclose(o, o2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(sf[:, :, 0], sf2, rtol=0, atol=1e-12)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_identical_slices_equal_dyadic(variant):
    """With k' = q' = 1/sqrt(E) * ones and equal gates on all slices every slice
    carries S/sqrt(E) of the dyadic state, so the output is the dyadic one."""
    rng = np.random.default_rng(3)
    E = 8
    d = rand_inputs(rng, E=E, with_s0=False)
    d["q2"] = np.full_like(d["q2"], 1 / np.sqrt(E))
    d["k2"] = np.full_like(d["k2"], 1 / np.sqrt(E))
    d["g"] = np.repeat(d["g"][..., :1], E, axis=-1)
    o, sf = run(variant, d)
    o2, sf2 = forms.dyadic(variant, d["q"], d["k"], d["v"], d["g"][..., 0], d["beta"])
    np.testing.assert_allclose(o, o2, rtol=0, atol=1e-12)
    for e in range(E):
        np.testing.assert_allclose(sf[:, :, e] * np.sqrt(E), sf2, rtol=0, atol=1e-12)


@pytest.mark.parametrize("with_beta", [True, False])
def test_quadratic_form_sgla(with_beta):
    """Eq. la3 parallel form with per-slice forgetting, brute force in T^2."""
    d = rand_inputs(np.random.default_rng(4), B=1, T=24, H=2, with_beta=with_beta)
    o, _ = run(SGLA, d)
    o2 = forms.quadratic_sgla(**d)
    np.testing.assert_allclose(o, o2, rtol=0, atol=1e-12)


def test_quadratic_form_slice_uniform_gates():
    """With one gate per token shared by all slices the read-out is
    sum_{s<=t} (prod of gates after s)(q2_t.k2_s)(q_t.k_s) v_s."""
    rng = np.random.default_rng(5)
    d = rand_inputs(rng, B=1, T=16, H=1, with_beta=False, with_s0=False)
    d["g"] = np.repeat(d["g"][..., :1], d["g"].shape[-1], axis=-1)
    o, _ = run(SGLA, d)
    a = np.exp(d["g"][0, :, 0, 0])
    T = o.shape[1]
    for t in range(T):
        ref = np.zeros(o.shape[-1])
        for s in range(t + 1):
            ref += (np.prod(a[s + 1:t + 1]) * (d["q2"][0, t, 0] @ d["k2"][0, s, 0])
                    * (d["q"][0, t, 0] @ d["k"][0, s, 0]) * d["v"][0, s, 0])
        np.testing.assert_allclose(o[0, t, 0], ref, rtol=0, atol=1e-12)


def test_gdn_reads_back_current_write():
    """Eq. gdn3 with beta = 1 and unit keys: reading with the writing keys returns
    exactly the value just written, whatever the state held before."""
    d = rand_inputs(np.random.default_rng(6), T=17)
    d["beta"] = np.ones_like(d["beta"])
    d["q"], d["q2"] = d["k"].copy(), d["k2"].copy()
    o, _ = run(GDN, d)
    np.testing.assert_allclose(o, d["v"], rtol=0, atol=1e-12)


def test_gdn_exact_retrieval_orthonormal_joint_keys():
    """Section 2.2: with orthonormal roles the third-order state stores E*K
    associations exactly.  Keys u_i (x) e_j, beta = 1: each probe returns the last
    value written under its pair, decayed by its slice's gates since the write
    (the probe's own gate included), and zero for pairs never written."""
    rng = np.random.default_rng(7)
    K, E, V = 4, 3, 5
    U = np.linalg.qr(rng.standard_normal((K, K)))[0]        # orthonormal u_i
    pairs = [(i, j) for i in range(K) for j in range(E)]
    order = [pairs[n] for n in rng.permutation(len(pairs))][:9]
    order += [order[2], order[5]]                           # overwrite two pairs
    probes = pairs
    T = len(order) + len(probes)
    q = np.zeros((1, T, 1, K)); k = np.zeros((1, T, 1, K)); v = np.zeros((1, T, 1, V))
    q2 = np.zeros((1, T, 1, E)); k2 = np.zeros((1, T, 1, E))
    g = rng.uniform(-0.2, 0.0, (1, T, 1, E))
    for t, (i, j) in enumerate(order):
        k[0, t, 0] = U[:, i]; k2[0, t, 0, j] = 1.0
        v[0, t, 0] = rng.standard_normal(V)
    for n, (i, j) in enumerate(probes):       # read-only probes: k = 0 writes nothing
        t = len(order) + n
        q[0, t, 0] = U[:, i]; q2[0, t, 0, j] = 1.0
    beta = np.ones((1, T, 1))
    o, _ = oracle.fwd(GDN, q, k, v, q2, k2, g, beta, None)
    a = np.exp(g[0, :, 0])
    for n, (i, j) in enumerate(probes):
        t = len(order) + n
        last = [s for s, p in enumerate(order) if p == (i, j)]
        if not last:
            expect = np.zeros(V)
        else:
            s = last[-1]
            expect = np.prod(a[s + 1:t + 1, j]) * v[0, s, 0]
        np.testing.assert_allclose(o[0, t, 0], expect, rtol=0, atol=1e-12)


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("chunk", [1, 2, 3, 4, 5, 8, 16, 21])
def test_chunkwise_equals_recurrent(variant, chunk):
    """Appendix A: the chunkwise form computes the recurrence exactly, for every
    chunk size including ones that do not divide T."""
    d = rand_inputs(np.random.default_rng(8), T=21, E=4, K=5, V=3)
    o, sf = run(variant, d)
    o2, sf2 = forms.chunkwise(variant, **d, chunk=chunk)
    np.testing.assert_allclose(o, o2, rtol=0, atol=1e-11)
    np.testing.assert_allclose(sf, sf2, rtol=0, atol=1e-11)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_chunkwise_strong_decay_no_overflow(variant):
    """Every decay factor is exp of a non-positive difference (Appendix A,
    numerical stability): gates of -1000 per token stay finite and exact."""
    d = rand_inputs(np.random.default_rng(9), T=19, E=3)
    d["g"][:, ::3] = -1000.0
    d["g"][:, 1::3] = np.log(2.0 ** -5)
    o, sf = run(variant, d)
    o2, sf2 = forms.chunkwise(variant, **d, chunk=8)
    assert np.all(np.isfinite(o2)) and np.all(np.isfinite(sf2))
    np.testing.assert_allclose(o, o2, rtol=0, atol=1e-11)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_zero_gate_limit(variant):
    """a -> 0 erases all history: o_t = (q2.k2)(q.k) beta v (retrieval is zero)."""
    d = rand_inputs(np.random.default_rng(10))
    d["g"] = np.full_like(d["g"], -800.0)
    o, sf = run(variant, d)
    coef = (np.einsum("bthe,bthe->bth", d["q2"], d["k2"]) *
            np.einsum("bthk,bthk->bth", d["q"], d["k"]) * d["beta"])
    np.testing.assert_allclose(o, coef[..., None] * d["v"], rtol=0, atol=1e-12)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_linearity_in_values_and_state(variant):
    """Both recurrences are linear in (v, s0) jointly."""
    rng = np.random.default_rng(11)
    d1 = rand_inputs(rng)
    d2 = dict(d1)
    d2["v"] = rng.standard_normal(d1["v"].shape)
    d2["s0"] = rng.standard_normal(d1["s0"].shape)
    d3 = dict(d1)
    d3["v"] = 2.0 * d1["v"] - 0.5 * d2["v"]
    d3["s0"] = 2.0 * d1["s0"] - 0.5 * d2["s0"]
    o1, s1 = run(variant, d1)
    o2, s2 = run(variant, d2)
    o3, s3 = run(variant, d3)
    np.testing.assert_allclose(o3, 2 * o1 - 0.5 * o2, rtol=0, atol=1e-12)
    np.testing.assert_allclose(s3, 2 * s1 - 0.5 * s2, rtol=0, atol=1e-12)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_resume_from_final_state(variant):
    d = rand_inputs(np.random.default_rng(12), T=20)
    o, sf = run(variant, d)
    cut = 7
    first = {kk: (x[:, :cut] if (x is not None and x.ndim >= 3 and kk != "s0") else x)
             for kk, x in d.items()}
    second = {kk: (x[:, cut:] if (x is not None and x.ndim >= 3 and kk != "s0") else x)
              for kk, x in d.items()}
    oa, sa = run(variant, first)
    second["s0"] = sa
    ob, sb = run(variant, second)
    np.testing.assert_allclose(np.concatenate([oa, ob], axis=1), o, rtol=0, atol=1e-13)
    np.testing.assert_allclose(sb, sf, rtol=0, atol=1e-13)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_step_repeated_equals_forward(variant):
    d = rand_inputs(np.random.default_rng(13), T=9)
    o, sf = run(variant, d)
    st = d["s0"].copy()
    for t in range(d["q"].shape[1]):
        ot, st = oracle.step(variant, d["q"][:, t], d["k"][:, t], d["v"][:, t],
                             d["q2"][:, t], d["k2"][:, t], d["g"][:, t],
                             None if d["beta"] is None else d["beta"][:, t], st)
        np.testing.assert_allclose(ot, o[:, t], rtol=0, atol=1e-13)
    np.testing.assert_allclose(st, sf, rtol=0, atol=1e-13)


def test_golden_worked_examples():
    """Hand-derived tiny cases (derivations in the fixture file)."""
    with open(os.path.join(HERE, "golden", "worked_examples.json")) as f:
        cases = json.load(f)["cases"]
    assert cases
    for c in cases:
        arr = lambda key: None if c[key] is None else np.array(c[key], dtype=np.float64)
        variant = {"sgla": SGLA, "gdn": GDN}[c["variant"]]
        o, sf = oracle.fwd(variant, arr("q"), arr("k"), arr("v"), arr("q2"), arr("k2"),
                           np.log(arr("a")), arr("beta"), arr("s0"))
        np.testing.assert_allclose(o, arr("o"), rtol=0, atol=1e-14, err_msg=c["name"])
        np.testing.assert_allclose(sf, arr("s_final"), rtol=0, atol=1e-14, err_msg=c["name"])

"""GPU parity of the backward (tla_bwd after a training tla_fwd) against the
oracle's fp64 reverse-mode recurrence, per gradient tensor, max|err|/RMS(ref)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36529_amd as tla
from paper_2609_36529_amd import synth
from helpers import TOL_BF16, TOL_F32, dev, host64, oracle_bwd_heads, rel_err

pytestmark = pytest.mark.gpu
SGLA, GDN = tla.SGLA, tla.GDN
GRADS = ("dq", "dk", "dv", "dq2", "dk2", "dg", "dbeta", "ds0")
NAMES = ("q", "k", "v", "q2", "k2", "g")


def cfg_of(variant, dtype, B=2, T=150, H=2, K=128, V=128, E=8, chunk=64, beta=None, s0=0.02, seed=9):
    if beta is None:
        beta = variant == GDN
    return synth.Config("t", variant, B, T, H, K, V, E, chunk, dtype, "softplus16", beta, s0, seed)


def run(cfg, inp, dO, dSf=None, grad_dtype=torch.float32):
    d = {k: dev(v) for k, v in inp.items()}
    _, _, saved = tla.fwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"],
                          d["s0"], chunk=cfg.chunk, out_dtype=torch.float32, training=True)
    gr = tla.bwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], d["s0"],
                 dev(dO), saved, dS_final=dev(dSf), chunk=cfg.chunk, out_dtype=grad_dtype)
    torch.cuda.synchronize()
    return gr


def check(cfg, tol, dS_final=False, seed_do=4):
    inp = synth.make_inputs(cfg)
    dO = synth.make_dO(cfg, seed=seed_do)
    dSf = None
    if dS_final:
        rng = np.random.default_rng(5)
        dSf = torch.from_numpy(rng.standard_normal((cfg.B, cfg.H, cfg.E, cfg.K, cfg.V))).float()
    gr = run(cfg, inp, dO, dSf)
    ref = oracle.bwd(cfg.variant, *[synth.to64(inp[n]) for n in NAMES], synth.to64(inp["beta"]),
                     synth.to64(inp["s0"]), synth.to64(dO), synth.to64(dSf))
    errs = {}
    for key in GRADS:
        if ref[key] is None:
            assert gr[key] is None
            continue
        got = host64(gr[key])
        assert np.all(np.isfinite(got)), key
        errs[key] = rel_err(got, ref[key])
    print(f"variant={cfg.variant} {cfg.dtype} T={cfg.T} C={cfg.chunk} E={cfg.E} K={cfg.K}: " +
          " ".join(f"{k}={v:.1e}" for k, v in errs.items()), flush=True)
    bad = {k: v for k, v in errs.items() if v > tol}
    assert not bad, bad


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("T", [150, 64, 1])
def test_f32_main_shape(variant, T):
    check(cfg_of(variant, "f32", T=T), TOL_F32, dS_final=True)


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("K,E,chunk", [(16, 4, 16), (32, 4, 32), (64, 8, 32), (128, 4, 64),
                                       (128, 1, 64), (128, 8, 32), (64, 16, 64), (32, 32, 32)])
def test_f32_shapes(variant, K, E, chunk):
    check(cfg_of(variant, "f32", T=77, K=K, V=K, E=E, chunk=chunk), TOL_F32, dS_final=True)


def test_sgla_with_beta_f32():
    check(cfg_of(SGLA, "f32", T=100, beta=True), TOL_F32, dS_final=True)


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("K,E,chunk", [(128, 8, 64), (128, 4, 64), (64, 8, 32), (16, 4, 16),
                                       (64, 16, 64), (32, 32, 32)])
def test_bf16_small(variant, K, E, chunk):
    check(cfg_of(variant, "bf16", T=203, K=K, V=K, E=E, chunk=chunk), TOL_BF16)


def test_bf16_E16():
    check(cfg_of(GDN, "bf16", T=150, E=16), TOL_BF16)


def test_bf16_sgla_with_beta():
    # zero final-state gradient, as in the GDN backward workload; a unit-scale
    # random dS_final with bf16 operands is covered in test_gpu_coverage.py
    check(cfg_of(SGLA, "bf16", T=170, beta=True), TOL_BF16)


def test_deterministic_bitwise():
    cfg = cfg_of(GDN, "bf16", T=300, H=4)
    inp = synth.make_inputs(cfg)
    dO = synth.make_dO(cfg)
    g1 = run(cfg, inp, dO)
    g2 = run(cfg, inp, dO)
    for key in GRADS:
        if g1[key] is not None:
            assert torch.equal(g1[key], g2[key]), key


def test_full_size_gdn_backward_sampled_heads():
    """GDN backward at B4 H8 T4096 K=V=128 E8 chunk 64 (bf16, upstream dO ~ N(0,1),
    zero final-state gradient), as launched by the bench; the oracle recomputes
    two sampled (b, h) heads over the whole sequence."""
    cfg = synth.CONFIGS["gdn_bf16"]
    inp = synth.make_inputs(cfg)
    dO = synth.make_dO(cfg)
    gr = run(cfg, inp, dO)
    heads = [(0, 0), (2, 7)]
    ref = oracle_bwd_heads(cfg.variant, inp, dO, heads)
    for (b, h), rg in ref.items():
        errs = {}
        for key in GRADS:
            got = host64(gr[key])
            got = got[b, h] if key == "ds0" else got[b, :, h]
            errs[key] = rel_err(got, rg[key])
        print(f"head {(b, h)}: " + " ".join(f"{k}={v:.1e}" for k, v in errs.items()), flush=True)
        bad = {k: v for k, v in errs.items() if v > TOL_BF16}
        assert not bad, bad
        bad = {k: v for k, v in errs.items() if v > TOL_BF16}
        assert not bad, bad


def test_gradient_matches_finite_differences_T64_slice():
    """Directional derivatives of the fp64 forward (central differences) on the
    first 64 tokens of head (0, 0) of the GDN workload match the GPU gradients."""
    cfg = synth.CONFIGS["gdn_bf16"]
    inp = synth.make_inputs(cfg, B=1, T=64, H=1)
    c1 = cfg_of(GDN, "bf16", B=1, T=64, H=1)
    dO = synth.make_dO(cfg, B=1, T=64, H=1)
    gr = run(c1, inp, dO)
    x = {n: synth.to64(inp[n]) for n in (*NAMES, "beta", "s0")}
    dO64 = synth.to64(dO)
    rng = np.random.default_rng(3)
    keys = {"q": "dq", "k": "dk", "v": "dv", "q2": "dq2", "k2": "dk2", "g": "dg", "beta": "dbeta",
            "s0": "ds0"}

    def loss(xx):
        o, _ = oracle.fwd(GDN, *[xx[n] for n in NAMES], xx["beta"], xx["s0"])
        return float(np.sum(o * dO64))
    for name, gk in keys.items():
        delta = rng.standard_normal(x[name].shape)
        h = 1e-6
        xp = dict(x); xp[name] = x[name] + h * delta
        xm = dict(x); xm[name] = x[name] - h * delta
        fd = (loss(xp) - loss(xm)) / (2 * h)
        an = float(np.sum(host64(gr[gk]) * delta))
        print(f"{name}: fd {fd:.6e} gpu {an:.6e}", flush=True)
        assert abs(fd - an) <= 2e-2 * max(abs(fd), 1e-3 * np.sqrt(delta.size)), (name, fd, an)


def test_bf16_gradient_outputs():
    """Gradients written in bf16 are the fp32 ones rounded once (within one ulp)."""
    cfg = cfg_of(GDN, "bf16", T=100)
    inp = synth.make_inputs(cfg)
    dO = synth.make_dO(cfg)
    g32 = run(cfg, inp, dO, grad_dtype=torch.float32)
    g16 = run(cfg, inp, dO, grad_dtype=torch.bfloat16)
    for key in ("dq", "dk", "dv", "dq2", "dk2"):
        assert g16[key].dtype == torch.bfloat16
        np.testing.assert_allclose(host64(g16[key]), host64(g32[key]), rtol=2 ** -8, atol=1e-6,
                                   err_msg=key)
    for key in ("dg", "dbeta", "ds0"):
        assert torch.equal(g16[key], g32[key]), key

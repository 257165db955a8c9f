"""GPU parity of the shapes and paths the main parity files do not reach:
value dimension different from the key dimension (the generality shapes of
the paper's Table 4 hold the value dimension at 128 while the key dimension
and E vary), a unit-scale final-state gradient with bf16 operands (a caller
that carries the state across calls), the binding's argument checks and the
autograd wrapper.  Errors are max|err| / RMS(ref) per tensor."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36529_amd as tla
from paper_2609_36529_amd import synth
from helpers import TOL_BF16, TOL_F32, dev, host64, rel_err

pytestmark = pytest.mark.gpu
SGLA, GDN = tla.SGLA, tla.GDN
NAMES = ("q", "k", "v", "q2", "k2", "g")
GRADS = ("dq", "dk", "dv", "dq2", "dk2", "dg", "dbeta", "ds0")


def cfg_of(variant, dtype, B=2, T=150, H=2, K=128, V=128, E=8, chunk=64, s0=0.02, seed=21):
    return synth.Config("cov", variant, B, T, H, K, V, E, chunk, dtype, "softplus16",
                        variant == GDN, s0, seed)


def fwd_bwd(cfg, inp, dO, dSf):
    d = {k: dev(v) for k, v in inp.items()}
    o, sf, saved = tla.fwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"],
                           d["s0"], chunk=cfg.chunk, out_dtype=torch.float32, training=True)
    gr = tla.bwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], d["s0"],
                 dev(dO), saved, dS_final=dev(dSf), chunk=cfg.chunk, out_dtype=torch.float32)
    torch.cuda.synchronize()
    return o, sf, gr


def check_fwd_bwd(cfg, tol, unit_dsf):
    inp = synth.make_inputs(cfg)
    dO = synth.make_dO(cfg, seed=31)
    dSf = None
    if unit_dsf:
        rng = np.random.default_rng(33)
        dSf = torch.from_numpy(rng.standard_normal((cfg.B, cfg.H, cfg.E, cfg.K, cfg.V))).float()
    o, sf, gr = fwd_bwd(cfg, inp, dO, dSf)
    args = [synth.to64(inp[n]) for n in NAMES] + [synth.to64(inp["beta"]), synth.to64(inp["s0"])]
    ro, rs = oracle.fwd(cfg.variant, *args)
    ref = oracle.bwd(cfg.variant, *args, synth.to64(dO), synth.to64(dSf))
    errs = {"o": rel_err(host64(o), ro), "s_final": rel_err(host64(sf), rs)}
    for key in GRADS:
        if ref[key] is None:
            assert gr[key] is None, key
            continue
        got = host64(gr[key])
        assert np.all(np.isfinite(got)), key
        errs[key] = rel_err(got, ref[key])
    print(f"variant={cfg.variant} {cfg.dtype} K={cfg.K} V={cfg.V} E={cfg.E} C={cfg.chunk} "
          f"T={cfg.T} dS_final={'unit' if unit_dsf else 'none'}: " +
          " ".join(f"{k}={v:.1e}" for k, v in errs.items()), flush=True)
    bad = {k: v for k, v in errs.items() if v > tol}
    assert not bad, bad


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("K,E,chunk", [(64, 16, 64), (32, 32, 32)])
def test_table4_shapes_value_dim_128(variant, dtype, K, E, chunk):
    """(K, E, chunk) = (64, 16, 64) and (32, 32, 32) with V = 128, forward and backward."""
    cfg = cfg_of(variant, dtype, B=1, T=133, K=K, V=128, E=E, chunk=chunk)
    check_fwd_bwd(cfg, TOL_F32 if dtype == "f32" else TOL_BF16, unit_dsf=(dtype == "f32"))


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_value_dim_smaller_than_key_dim(variant, dtype):
    cfg = cfg_of(variant, dtype, B=1, T=97, K=128, V=64, E=8, chunk=64)
    check_fwd_bwd(cfg, TOL_F32 if dtype == "f32" else TOL_BF16, unit_dsf=(dtype == "f32"))


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_forward_value_dim_256(variant, dtype):
    """The forward at V = 256 (sixteen value tiles per head)."""
    cfg = cfg_of(variant, dtype, B=1, T=170, K=128, V=256, E=8, chunk=64)
    inp = synth.make_inputs(cfg)
    d = {k: dev(v) for k, v in inp.items()}
    o, sf, _ = tla.fwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"],
                       d["s0"], chunk=cfg.chunk, out_dtype=torch.float32)
    torch.cuda.synchronize()
    ro, rs = oracle.fwd(cfg.variant, *[synth.to64(inp[n]) for n in NAMES], synth.to64(inp["beta"]),
                        synth.to64(inp["s0"]))
    eo, es = rel_err(host64(o), ro), rel_err(host64(sf), rs)
    print(f"V=256 variant={variant} {dtype}: o err {eo:.2e} s_final err {es:.2e}", flush=True)
    tol = TOL_F32 if dtype == "f32" else TOL_BF16
    assert eo <= tol and es <= tol


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_bf16_backward_unit_final_state_gradient(variant):
    """bf16 operands with a unit-scale random final-state gradient (a caller
    that carries the state across calls)."""
    cfg = cfg_of(variant, "bf16", B=2, T=203, H=2, E=8)
    check_fwd_bwd(cfg, TOL_BF16, unit_dsf=True)


def test_binding_rejects_bad_arguments_before_launch():
    cfg = cfg_of(GDN, "bf16", B=1, T=64, H=2)
    inp = synth.make_inputs(cfg)
    d = {k: dev(v) for k, v in inp.items()}
    args = [d[n] for n in NAMES] + [d["beta"], d["s0"]]
    bad_k = d["k"][:, :32].contiguous()
    with pytest.raises(ValueError, match="k has shape"):
        tla.fwd(GDN, d["q"], bad_k, *args[2:])
    with pytest.raises(ValueError, match="contiguous"):
        tla.fwd(GDN, d["q"], d["k"].transpose(1, 2), *args[2:])
    with pytest.raises(TypeError, match="g must be"):
        tla.fwd(GDN, *args[:5], d["g"].to(torch.bfloat16), *args[6:])
    with pytest.raises(ValueError, match="s0 has shape"):
        tla.fwd(GDN, *args[:7], d["s0"][:, :1].contiguous())
    _, _, saved = tla.fwd(GDN, *args, training=True)
    dO = dev(synth.make_dO(cfg))
    with pytest.raises(ValueError, match="saved holds"):
        tla.bwd(GDN, *args, dO, saved[: saved.numel() // 2])
    with pytest.raises(ValueError, match="dO has shape"):
        tla.bwd(GDN, *args, dO[:, :10].contiguous(), saved)
    with pytest.raises(TypeError, match="q2 must be"):
        tla.bwd(GDN, *args[:3], d["q2"].float(), *args[4:], dO, saved)
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(ValueError, match="ws holds"):
        tla.bwd(GDN, *args, dO, saved, ws=small)
    with pytest.raises(ValueError, match="ws holds"):
        tla.fwd(GDN, *args, ws=small)
    torch.cuda.synchronize()


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_autograd_wrapper_matches_bwd(variant):
    """tla.attention under torch.autograd gives the gradients of tla.bwd
    (bitwise: the same kernels) and they match the oracle."""
    cfg = cfg_of(variant, "f32", B=1, T=100, H=2)
    inp = synth.make_inputs(cfg)
    leaves = {n: dev(inp[n]).requires_grad_(True) for n in NAMES}
    beta = None if inp["beta"] is None else dev(inp["beta"]).requires_grad_(True)
    s0 = dev(inp["s0"]).requires_grad_(True)
    o, sf = tla.attention(variant, *[leaves[n] for n in NAMES], beta, s0, chunk=64)
    dO = dev(synth.make_dO(cfg, seed=41))
    wf = torch.randn(sf.shape, generator=torch.Generator().manual_seed(43)).cuda()
    loss = (o * dO).sum() + (sf * wf).sum()
    loss.backward()
    d = {k: dev(v) for k, v in inp.items()}
    _, _, saved = tla.fwd(variant, *[d[n] for n in NAMES], d["beta"], d["s0"], chunk=64, training=True)
    ref = tla.bwd(variant, *[d[n] for n in NAMES], d["beta"], d["s0"], dO, saved, dS_final=wf, chunk=64)
    torch.cuda.synchronize()
    for n in NAMES:
        assert torch.equal(leaves[n].grad, ref["d" + n]), n
    assert torch.equal(s0.grad, ref["ds0"])
    if beta is not None:
        assert torch.equal(beta.grad, ref["dbeta"])
    rg = oracle.bwd(variant, *[synth.to64(inp[n]) for n in NAMES], synth.to64(inp["beta"]),
                    synth.to64(inp["s0"]), synth.to64(dO.cpu()), synth.to64(wf.cpu()))
    for n in NAMES:
        assert rel_err(host64(leaves[n].grad), rg["d" + n]) <= TOL_F32, n


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("V,T,s0", [(128, 150, 0.02), (64, 77, 0.0), (256, 200, 0.02)])
def test_e16_inference_forward(variant, V, T, s0):
    """E = 16, K = 128, chunk 64 with bf16 operands: the inference forward
    (two key slices per accumulator tile, 8 value columns per workgroup) and
    the training forward (16 columns per workgroup) against the oracle."""
    cfg = cfg_of(variant, "bf16", B=1, T=T, H=3, K=128, V=V, E=16, chunk=64, s0=s0, seed=23)
    inp = synth.make_inputs(cfg)
    d = {k: dev(v) for k, v in inp.items()}
    args = [d[n] for n in NAMES] + [d["beta"], d["s0"]]
    o, sf, _ = tla.fwd(variant, *args, chunk=64, out_dtype=torch.float32)
    o_t, sf_t, _ = tla.fwd(variant, *args, chunk=64, out_dtype=torch.float32, training=True)
    torch.cuda.synchronize()
    ro, rs = oracle.fwd(variant, *[synth.to64(inp[n]) for n in NAMES], synth.to64(inp["beta"]),
                        synth.to64(inp["s0"]))
    errs = {"o": rel_err(host64(o), ro), "s_final": rel_err(host64(sf), rs),
            "o_train": rel_err(host64(o_t), ro), "s_final_train": rel_err(host64(sf_t), rs)}
    print(f"E16 variant={variant} V={V} T={T}: " + " ".join(f"{k}={v:.1e}" for k, v in errs.items()),
          flush=True)
    assert all(v <= TOL_BF16 for v in errs.values()), errs


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("E", [1, 2, 4, 8, 16])
def test_head_dim_16_instances(variant, dtype, E):
    """K = V = 16, chunk 16 (the MQAR model's heads) at every E of its sweep."""
    cfg = cfg_of(variant, dtype, B=2, T=45, H=3, K=16, V=16, E=E, chunk=16, seed=29)
    check_fwd_bwd(cfg, TOL_F32 if dtype == "f32" else TOL_BF16, unit_dsf=(dtype == "f32"))

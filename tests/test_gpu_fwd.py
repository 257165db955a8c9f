"""GPU parity of the chunkwise forward and the decode step against the fp64
oracle (max|err| / RMS(ref) per output tensor), through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36529_amd as tla
from paper_2609_36529_amd import synth
from helpers import TOL_BF16, TOL_F32, dev, host64, oracle_fwd_heads, rel_err

pytestmark = pytest.mark.gpu
SGLA, GDN = tla.SGLA, tla.GDN


def small_cfg(variant, dtype, B=2, T=200, H=2, K=128, V=128, E=8, chunk=64, s0=0.02,
              gate="softplus16", seed=7):
    return synth.Config("t", variant, B, T, H, K, V, E, chunk, dtype, gate,
                        variant == GDN, s0, seed)


def run_fwd(cfg, inp, out_dtype=torch.float32, training=False):
    d = {k: dev(v) for k, v in inp.items()}
    o, sf, saved = tla.fwd(cfg.variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"],
                           d["s0"], chunk=cfg.chunk, out_dtype=out_dtype, training=training)
    torch.cuda.synchronize()
    return o, sf, saved


def check_all_heads(cfg, inp, tol, out_dtype=torch.float32):
    o, sf, _ = run_fwd(cfg, inp, out_dtype)
    oo, ss = oracle.fwd(cfg.variant, *[synth.to64(inp[n]) for n in ("q", "k", "v", "q2", "k2", "g")],
                        synth.to64(inp["beta"]), synth.to64(inp["s0"]))
    eo, es = rel_err(host64(o), oo), rel_err(host64(sf), ss)
    print(f"{cfg.variant=} {cfg.dtype=} T={cfg.T} C={cfg.chunk} E={cfg.E} K={cfg.K}: "
          f"o err {eo:.2e}  s_final err {es:.2e}", flush=True)
    assert np.all(np.isfinite(host64(o)))
    assert eo <= tol and es <= tol, (eo, es)


def test_tiny_sgla_f32_config():
    """The tiny fp32 sGLA workload: B1 H1 T64 K16 E4 V16 chunk 16."""
    cfg = synth.CONFIGS["tiny_sgla_f32"]
    check_all_heads(cfg, synth.make_inputs(cfg), TOL_F32)


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("T", [200, 64, 1, 37])
def test_f32_operands_main_shape(variant, T):
    """fp32 operands through the same kernels at K=V=128, E=8, chunk 64
    (several chunks plus a ragged tail, a single chunk, one token)."""
    cfg = small_cfg(variant, "f32", T=T)
    check_all_heads(cfg, synth.make_inputs(cfg), TOL_F32)


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("K,E,chunk", [(128, 8, 64), (128, 4, 64), (128, 1, 64), (64, 8, 32),
                                       (32, 4, 32), (16, 4, 16), (128, 8, 32), (64, 16, 64),
                                       (32, 32, 32)])
def test_bf16_small(variant, K, E, chunk):
    cfg = small_cfg(variant, "bf16", T=203, K=K, V=K, E=E, chunk=chunk)
    check_all_heads(cfg, synth.make_inputs(cfg), TOL_BF16)


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("K,E,chunk", [(64, 16, 64), (32, 32, 32)])
def test_f32_wide_second_keys(variant, K, E, chunk):
    """The generality shapes of the paper's Table 4 (E = 16 at K = 64,
    E = 32 at K = 32) with fp32 operands."""
    cfg = small_cfg(variant, "f32", B=1, T=97, H=2, K=K, V=K, E=E, chunk=chunk)
    check_all_heads(cfg, synth.make_inputs(cfg), TOL_F32)


def test_bf16_E16():
    cfg = small_cfg(GDN, "bf16", T=150, H=2, E=16)
    check_all_heads(cfg, synth.make_inputs(cfg), TOL_BF16)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_sgla_with_beta_and_nonneg_second_keys(variant):
    cfg = small_cfg(variant, "bf16", T=130)
    cfg.beta = True
    check_all_heads(cfg, synth.make_inputs(cfg, nonneg_second=True), TOL_BF16)


@pytest.mark.parametrize("variant", [SGLA, GDN])
def test_extreme_gates_finite(variant):
    """Log-gates of -1000 and log(2^-5) per token (Appendix A numerics; half-lives
    down to 0.2 tokens, Appendix B) stay finite and match the oracle."""
    cfg = small_cfg(variant, "f32", T=150)
    inp = synth.make_inputs(cfg)
    g = inp["g"].clone()
    g[:, ::5] = -1000.0
    g[:, 1::5] = float(np.log(2.0 ** -5))
    inp["g"] = g
    check_all_heads(cfg, inp, TOL_F32)


@pytest.mark.parametrize("name", ["sgla_bf16", "gdn_bf16"])
def test_full_size_sampled_heads(name):
    """The B4 H8 T4096 K=V=128 E8 chunk-64 workloads, as launched by the bench;
    the oracle recomputes two sampled (b, h) heads over the whole sequence."""
    cfg = synth.CONFIGS[name]
    inp = synth.make_inputs(cfg)
    o, sf, _ = run_fwd(cfg, inp)
    heads = [(0, 0), (3, 5)]
    ref = oracle_fwd_heads(cfg.variant, inp, heads)
    o64, sf64 = host64(o), host64(sf)
    for (b, h), (ro, rs) in ref.items():
        eo, es = rel_err(o64[b, :, h], ro), rel_err(sf64[b, h], rs)
        print(f"{name} head {(b, h)}: o err {eo:.2e} s_final err {es:.2e}", flush=True)
        assert eo <= TOL_BF16 and es <= TOL_BF16, (eo, es)
    assert np.all(np.isfinite(o64))


def test_long_context_E16_sampled_prefix():
    """GDN at E=16, H=16, B=1, T=65536, chunk 64 (1024 chunks carried by one
    launch).  Outputs at t < 4096 do not depend on later positions, so the
    oracle recomputes that prefix for two sampled heads; the final state is
    checked by resuming: [0, T/2) then [T/2, T) from the returned mid state
    gives the same s_final as the single launch."""
    cfg = synth.CONFIGS["gdn_long_bf16"]
    inp = synth.make_inputs(cfg)
    o, sf, _ = run_fwd(cfg, inp)
    P = 4096
    pre = {k: (None if v is None or k == "s0" else v[:, :P]) for k, v in inp.items()}
    pre["s0"] = inp["s0"]
    ref = oracle_fwd_heads(cfg.variant, pre, [(0, 0), (0, 11)])
    o64 = host64(o)
    assert np.all(np.isfinite(o64))
    for (b, h), (ro, _) in ref.items():
        eo = rel_err(o64[b, :P, h], ro)
        print(f"long context head {(b, h)}: prefix o err {eo:.2e}", flush=True)
        assert eo <= TOL_BF16, eo
    half = cfg.T // 2
    first = {k: (None if v is None or k == "s0" else v[:, :half]) for k, v in inp.items()}
    first["s0"] = inp["s0"]
    _, mid, _ = run_fwd(cfg, first)
    second = {k: (None if v is None or k == "s0" else v[:, half:]) for k, v in inp.items()}
    second["s0"] = mid.cpu()
    o2, sf2, _ = run_fwd(cfg, second)
    es = rel_err(host64(sf2), host64(sf))
    eo2 = rel_err(host64(o2), o64[:, half:])
    print(f"long context resume: s_final err {es:.2e}, second-half o err {eo2:.2e}", flush=True)
    assert es <= 1e-6 and eo2 <= 1e-6, (es, eo2)


def test_bf16_output_dtype():
    cfg = small_cfg(GDN, "bf16", T=100)
    inp = synth.make_inputs(cfg)
    o16, _, _ = run_fwd(cfg, inp, out_dtype=torch.bfloat16)
    o32, _, _ = run_fwd(cfg, inp, out_dtype=torch.float32)
    assert o16.dtype == torch.bfloat16
    # o rounded to bf16: within one bf16 ulp of the fp32 output
    np.testing.assert_allclose(host64(o16), host64(o32), rtol=2 ** -8, atol=1e-6)


def test_deterministic_bitwise():
    cfg = small_cfg(GDN, "bf16", T=300, H=4)
    inp = synth.make_inputs(cfg)
    o1, s1, _ = run_fwd(cfg, inp)
    o2, s2, _ = run_fwd(cfg, inp)
    assert torch.equal(o1, o2) and torch.equal(s1, s2)


def test_resume_and_in_place_state():
    """fwd(0:T) equals fwd(T1:T) from fwd(0:T1)'s final state; s_final may alias s0."""
    cfg = small_cfg(GDN, "f32", T=192)
    inp = synth.make_inputs(cfg)
    d = {k: dev(v) for k, v in inp.items()}
    o, sf, _ = tla.fwd(GDN, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], d["s0"])
    cut = 128
    part = lambda x, a, b: x[:, a:b].contiguous()
    st = d["s0"].clone()
    oa, _, _ = tla.fwd(GDN, *[part(d[n], 0, cut) for n in ("q", "k", "v", "q2", "k2", "g", "beta")],
                       st, s_final=st)
    ob, _, _ = tla.fwd(GDN, *[part(d[n], cut, 192) for n in ("q", "k", "v", "q2", "k2", "g", "beta")],
                       st, s_final=st)
    torch.cuda.synchronize()
    assert rel_err(host64(torch.cat([oa, ob], 1)), host64(o)) < 1e-5
    assert rel_err(host64(st), host64(sf)) < 1e-5


def test_empty_sequence_passes_state_through():
    cfg = small_cfg(GDN, "bf16", T=0)
    inp = synth.make_inputs(cfg)
    o, sf, _ = run_fwd(cfg, inp)
    assert o.numel() == 0
    assert torch.equal(sf.cpu(), inp["s0"])


def test_chunk_sizes_agree():
    cfg = small_cfg(GDN, "f32", T=256)
    inp = synth.make_inputs(cfg)
    cfg.chunk = 64
    o64, s64, _ = run_fwd(cfg, inp)
    cfg.chunk = 32
    o32, s32, _ = run_fwd(cfg, inp)
    assert rel_err(host64(o32), host64(o64)) < 1e-5
    assert rel_err(host64(s32), host64(s64)) < 1e-5


# ------------------------------------------------------------------ decode
def step_inputs(N, H, K, V, E, dtype, variant, seed):
    tok = synth.make_decode_token(N, H, K, V, E, dtype=dtype, seed=seed, variant=variant)
    return tok


@pytest.mark.parametrize("variant", [SGLA, GDN])
@pytest.mark.parametrize("dtype,K,V,E", [("f32", 16, 16, 4), ("f32", 128, 128, 8),
                                         ("bf16", 128, 128, 16), ("bf16", 128, 128, 1),
                                         ("bf16", 32, 48, 4), ("f32", 64, 64, 16),
                                         ("bf16", 32, 32, 32)])
def test_step_matches_oracle(variant, dtype, K, V, E):
    N, H = 3, 2
    state = synth.make_decode_state(N, H, E, K, V, seed=11)
    st_dev = dev(state)
    ref_state = synth.to64(state)
    for it in range(3):
        tok = step_inputs(N, H, K, V, E, dtype, variant, seed=100 + it)
        d = {k: dev(v) for k, v in tok.items()}
        o = tla.step(variant, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], st_dev,
                     out_dtype=torch.float32)
        torch.cuda.synchronize()
        ro, ref_state = oracle.step(variant, *[synth.to64(tok[n]) for n in
                                               ("q", "k", "v", "q2", "k2", "g")],
                                    synth.to64(tok["beta"]), ref_state)
        eo, es = rel_err(host64(o), ro), rel_err(host64(st_dev), ref_state)
        print(f"step {it}: o err {eo:.2e} state err {es:.2e}", flush=True)
        assert eo <= TOL_F32 and es <= TOL_F32, (eo, es)


def test_step_repeated_equals_chunkwise_forward():
    """T decode steps reproduce the chunkwise forward (recurrent = chunkwise)."""
    cfg = small_cfg(GDN, "f32", B=2, T=40, H=2)
    inp = synth.make_inputs(cfg)
    o, sf, _ = run_fwd(cfg, inp)
    st = dev(inp["s0"]).clone()
    outs = []
    for t in range(cfg.T):
        tok = {n: dev(inp[n][:, t]) for n in ("q", "k", "v", "q2", "k2", "g", "beta")}
        outs.append(tla.step(GDN, tok["q"], tok["k"], tok["v"], tok["q2"], tok["k2"], tok["g"],
                             tok["beta"], st, out_dtype=torch.float32))
    torch.cuda.synchronize()
    assert rel_err(host64(torch.stack(outs, 1)), host64(o)) < 1e-5
    assert rel_err(host64(st), host64(sf)) < 1e-5


def test_decode_batch256_sampled():
    """Decode at N=256, H=16, E=16, K=V=128 (4 GiB fp32 state): 3 steps on the
    full batch, the oracle follows 4 sampled sequences."""
    N, H, E, K, V = 256, 16, 16, 128, 128
    state = synth.make_decode_state(N, H, E, K, V)
    st_dev = dev(state)
    pick = [0, 77, 128, 255]
    ref_state = synth.to64(state[pick])
    del state
    for it in range(3):
        tok = synth.make_decode_token(N, H, K, V, E, dtype="bf16", seed=500 + it)
        d = {k: dev(v) for k, v in tok.items()}
        o = tla.step(GDN, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], st_dev,
                     out_dtype=torch.float32)
        torch.cuda.synchronize()
        ro, ref_state = oracle.step(GDN, *[synth.to64(tok[n][pick]) for n in
                                           ("q", "k", "v", "q2", "k2", "g")],
                                    synth.to64(tok["beta"][pick]), ref_state)
        eo = rel_err(host64(o[pick]), ro)
        es = rel_err(host64(st_dev[pick]), ref_state)
        print(f"decode step {it}: o err {eo:.2e} state err {es:.2e}", flush=True)
        assert eo <= TOL_F32 and es <= TOL_F32

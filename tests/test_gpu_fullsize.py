"""Whole-tensor GPU parity at the configuration shapes (every head, every
position, every gradient), against the fp64 oracle run on all heads in one
call (OpenMP over heads):
  * sGLA and GDN inference forwards at B4 H8 T4096 K=V=128 E8 chunk 64
    (outputs and final states of all 32 heads);
  * the GDN backward on the same inputs (all 8 gradients, all 32 heads),
    with a zero and with a unit-scale final-state gradient, and the sGLA
    backward on the sGLA inputs;
  * the long-context GDN forward at B1 H16 T65536 E16 (all 16 heads, the
    whole output and the final state);
  * the decode step at N256 H16 E16: 1000 steps on 8 sequences followed by
    the oracle step by step, and 10 steps on all 256 sequences.
Errors are max|err| / RMS(ref) per tensor (bf16 operands: 2e-2; decode
carries an fp32 state from bf16 tokens: 1e-5)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36529_amd as tla
from paper_2609_36529_amd import synth
from helpers import TOL_BF16, TOL_F32, host64, rel_err

pytestmark = pytest.mark.gpu
NAMES = ("q", "k", "v", "q2", "k2", "g")


def _dev(inp):
    return {k: (None if v is None else v.cuda()) for k, v in inp.items()}


def _oracle_args(inp):
    return [synth.to64(inp[n]) for n in NAMES] + [synth.to64(inp["beta"]), synth.to64(inp["s0"])]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["sgla_bf16", "gdn_bf16"])
def test_forward_all_heads(name):
    cfg = synth.CONFIGS[name]
    inp = synth.make_inputs(cfg)
    d = _dev(inp)
    o, sf, _ = tla.fwd(cfg.variant, *[d[n] for n in NAMES], d["beta"], d["s0"], chunk=cfg.chunk,
                       out_dtype=torch.float32)
    torch.cuda.synchronize()
    ro, rs = oracle.fwd(cfg.variant, *_oracle_args(inp))
    eo, es = rel_err(host64(o), ro), rel_err(host64(sf), rs)
    print(f"{name} all heads: o err {eo:.2e}  s_final err {es:.2e} "
          f"(oracle on {oracle.num_threads()} threads)", flush=True)
    assert np.all(np.isfinite(host64(o)))
    assert eo <= TOL_BF16 and es <= TOL_BF16, (eo, es)


def _backward_all_heads(with_final_state_gradient, name="gdn_bf16"):
    cfg = synth.CONFIGS[name]
    inp = synth.make_inputs(cfg)
    dO = synth.make_dO(cfg)
    dSf = None
    if with_final_state_gradient:
        rng = np.random.default_rng(17)
        dSf = torch.from_numpy(rng.standard_normal((cfg.B, cfg.H, cfg.E, cfg.K, cfg.V))).float()
    d = _dev(inp)
    _, _, saved = tla.fwd(cfg.variant, *[d[n] for n in NAMES], d["beta"], d["s0"], chunk=cfg.chunk,
                          out_dtype=torch.float32, training=True)
    gr = tla.bwd(cfg.variant, *[d[n] for n in NAMES], d["beta"], d["s0"], dO.cuda(), saved,
                 dS_final=None if dSf is None else dSf.cuda(), chunk=cfg.chunk,
                 out_dtype=torch.float32)
    torch.cuda.synchronize()
    ref = oracle.bwd(cfg.variant, *_oracle_args(inp), synth.to64(dO),
                     None if dSf is None else synth.to64(dSf))
    errs = {}
    for key in ("dq", "dk", "dv", "dq2", "dk2", "dg", "dbeta", "ds0"):
        if ref[key] is None:  # sGLA without beta
            assert gr[key] is None, key
            continue
        got = host64(gr[key])
        assert np.all(np.isfinite(got)), key
        errs[key] = rel_err(got, ref[key])
    label = "with unit final-state gradient" if with_final_state_gradient else ""
    print(f"{name} backward all heads{' ' + label if label else ''}: " + " ".join(f"{k}={v:.1e}" for k, v in errs.items()),
          flush=True)
    bad = {k: v for k, v in errs.items() if v > TOL_BF16}
    assert not bad, bad


@pytest.mark.timeout(900)
def test_gdn_backward_all_heads():
    """The GDN backward workload: dO ~ N(0, 1) bf16, zero final-state gradient."""
    _backward_all_heads(False)


@pytest.mark.timeout(900)
def test_gdn_backward_all_heads_with_final_state_gradient():
    """The same backward when the caller carries state on: a unit-scale
    dS_final ~ N(0, 1) (the chunk-end state gradients then travel as bf16
    (hi, lo) pairs)."""
    _backward_all_heads(True)


@pytest.mark.timeout(900)
def test_sgla_backward_all_heads():
    """The sGLA backward on the sGLA forward workload's inputs (B4 H8 T4096
    E8 bf16), zero final-state gradient."""
    _backward_all_heads(False, "sgla_bf16")


@pytest.mark.timeout(900)
def test_long_context_all_heads_whole_sequence():
    """GDN B1 H16 T65536 E16 chunk 64 (1024 chunks carried by one launch):
    every output position and the final state of all 16 heads."""
    cfg = synth.CONFIGS["gdn_long_bf16"]
    inp = synth.make_inputs(cfg)
    d = _dev(inp)
    o, sf, _ = tla.fwd(cfg.variant, *[d[n] for n in NAMES], d["beta"], d["s0"], chunk=cfg.chunk,
                       out_dtype=torch.float32)
    torch.cuda.synchronize()
    o64, sf64 = host64(o), host64(sf)
    del o, sf, d
    ro, rs = oracle.fwd(cfg.variant, *_oracle_args(inp))
    eo, es = rel_err(o64, ro), rel_err(sf64, rs)
    print(f"long context all heads: o err {eo:.2e}  s_final err {es:.2e}", flush=True)
    assert np.all(np.isfinite(o64))
    assert eo <= TOL_BF16 and es <= TOL_BF16, (eo, es)


@pytest.mark.timeout(900)
def test_decode_1000_steps_on_8_sequences():
    """tla_step on the full N256 H16 E16 batch for 1000 steps (fresh bf16
    tokens each step, fp32 state in place); the oracle follows 8 sequences
    step by step (outputs every step, states at the end)."""
    N, H, E, K, V = 256, 16, 16, 128, 128
    pick = [0, 1, 77, 128, 129, 200, 254, 255]
    state = synth.make_decode_state(N, H, E, K, V)
    st_dev = state.cuda()
    ref_state = synth.to64(state[pick])
    del state
    worst = 0.0
    for it in range(1000):
        tok = synth.make_decode_token(N, H, K, V, E, dtype="bf16", seed=10_000 + it)
        d = {k: v.cuda() for k, v in tok.items()}
        o = tla.step(tla.GDN, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], st_dev,
                     out_dtype=torch.float32)
        ro, ref_state = oracle.step(tla.GDN, *[synth.to64(tok[n][pick]) for n in NAMES],
                                    synth.to64(tok["beta"][pick]), ref_state)
        worst = max(worst, rel_err(host64(o[pick]), ro))
        if it % 200 == 199:
            print(f"decode step {it + 1}: worst o err so far {worst:.2e}", flush=True)
    es = rel_err(host64(st_dev[pick]), ref_state)
    print(f"decode 1000 steps: o err {worst:.2e}, state err {es:.2e}", flush=True)
    assert worst <= TOL_F32 and es <= TOL_F32, (worst, es)


@pytest.mark.timeout(900)
def test_decode_10_steps_all_256_sequences():
    N, H, E, K, V = 256, 16, 16, 128, 128
    state = synth.make_decode_state(N, H, E, K, V)
    st_dev = state.cuda()
    ref_state = synth.to64(state)
    del state
    for it in range(10):
        tok = synth.make_decode_token(N, H, K, V, E, dtype="bf16", seed=20_000 + it)
        d = {k: v.cuda() for k, v in tok.items()}
        o = tla.step(tla.GDN, d["q"], d["k"], d["v"], d["q2"], d["k2"], d["g"], d["beta"], st_dev,
                     out_dtype=torch.float32)
        ro, ref_state = oracle.step(tla.GDN, *[synth.to64(tok[n]) for n in NAMES],
                                    synth.to64(tok["beta"]), ref_state)
        eo = rel_err(host64(o), ro)
        print(f"decode all 256, step {it + 1}: o err {eo:.2e}", flush=True)
        assert eo <= TOL_F32, eo
    # final states, compared in blocks of sequences (the fp64 copy is 8.6 GB)
    rms = np.sqrt(np.mean(ref_state * ref_state))
    worst = 0.0
    for n0 in range(0, N, 32):
        got = host64(st_dev[n0:n0 + 32])
        worst = max(worst, float(np.max(np.abs(got - ref_state[n0:n0 + 32]))))
    es = worst / rms
    print(f"decode all 256, 10 steps: state err {es:.2e}", flush=True)
    assert es <= TOL_F32, es

"""Shared test utilities: error metric, device transfer, oracle on sampled heads."""
import numpy as np
import torch

import oracle
from paper_2609_36529_amd import synth

# max|err| / RMS(ref) bounds: fp32 operands and bf16 operands (fp32 accumulation)
TOL_F32 = 1e-5
TOL_BF16 = 2e-2


def rel_err(got, ref):
    """max |got - ref| / RMS(ref), computed in float64."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    rms = np.sqrt(np.mean(ref * ref))
    if rms == 0.0:
        return float(np.max(np.abs(got - ref))) if got.size else 0.0
    return float(np.max(np.abs(got - ref)) / rms)


def dev(x, device="cuda"):
    return None if x is None else x.to(device).contiguous()


def host64(x):
    return None if x is None else x.detach().to("cpu", torch.float64).numpy()


def _stack(x, heads):
    """Selected (b, h) slices of a [B,T,H,...] tensor stacked as [n,T,1,...] float64."""
    if x is None:
        return None
    return np.stack([synth.to64(x[b, :, h:h + 1]) for (b, h) in heads])


def _stack_state(x, heads):
    if x is None:
        return None
    return np.stack([synth.to64(x[b, h:h + 1]) for (b, h) in heads])


def oracle_fwd_heads(variant, inp, heads):
    """Oracle forward on selected (b, h) pairs (one call, OpenMP over them);
    returns {(b,h): (o [T,V], sf [E,K,V])}."""
    args = [_stack(inp[n], heads) for n in ("q", "k", "v", "q2", "k2", "g")]
    o, sf = oracle.fwd(variant, *args, _stack(inp["beta"], heads), _stack_state(inp["s0"], heads))
    return {bh: (o[i, :, 0], sf[i, 0]) for i, bh in enumerate(heads)}


def oracle_bwd_heads(variant, inp, dO, heads, dS_final=None):
    args = [_stack(inp[n], heads) for n in ("q", "k", "v", "q2", "k2", "g")]
    gr = oracle.bwd(variant, *args, _stack(inp["beta"], heads), _stack_state(inp["s0"], heads),
                    _stack(dO, heads), _stack_state(dS_final, heads))
    out = {}
    for i, bh in enumerate(heads):
        out[bh] = {k: (None if v is None else (v[i, 0] if k == "ds0" else v[i, :, 0]))
                   for k, v in gr.items()}
    return out

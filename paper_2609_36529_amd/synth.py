"""Seeded synthetic inputs for triadic linear attention.

This module holds no arithmetic of the operator: it only draws random inputs
with the shapes and distributions of the paper's language-model workloads
(head dimension 128, second-key dimension E, 4k pretraining and 64k extension
contexts; Section 3.1 and Appendix D) and casts them to the requested dtype.
Both the GPU path and the fp64 oracle are fed from what it returns; the oracle
consumes the already-cast values.

Conventions (all from a ``numpy.random.Generator(PCG64(seed))`` in fp64):
* q, k, q2, k2 ~ N(0, 1), then L2-normalised per vector (Alg. 2 normalises
  q, k, q', k'); optional ``nonneg_second`` applies softplus to q2, k2 before
  normalising (the softplus activation of Alg. 2).
* v ~ N(0, 1); dO ~ N(0, 1).
* log-gates g = log a <= 0 per slice, one of the recipes below.
* beta = sigmoid(N(0, 1)) for GDN, None for plain sGLA.
* initial state ~ N(0, std^2) in fp32, or None for a zero state.
"""
from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

SGLA, GDN = 0, 1


@dataclass
class Config:
    name: str
    variant: int
    B: int
    T: int
    H: int
    K: int
    V: int
    E: int
    chunk: int
    dtype: str                   # "f32" or "bf16": q, k, v, q2, k2, dO
    gate: str                    # "logsigmoid_n3" or "softplus16"
    beta: bool                   # GDN always True
    s0_std: float                # 0 -> zero initial state
    seed: int
    notes: str = ""
    extra: dict = field(default_factory=dict)


# The workloads: tiny fp32 sGLA; sGLA and GDN at the 400M/1.3B head shape
# (B=4, H=8, T=4096, K=V=128, E=8); a 64k-token GDN at E=16; decode at E=16.
CONFIGS = {
    "tiny_sgla_f32": Config("tiny_sgla_f32", SGLA, 1, 64, 1, 16, 16, 4, 16, "f32",
                            "logsigmoid_n3", False, 0.0, 101),
    "sgla_bf16": Config("sgla_bf16", SGLA, 4, 4096, 8, 128, 128, 8, 64, "bf16",
                        "softplus16", False, 0.0, 102),
    "gdn_bf16": Config("gdn_bf16", GDN, 4, 4096, 8, 128, 128, 8, 64, "bf16",
                       "softplus16", True, 0.02, 103),
    "gdn_long_bf16": Config("gdn_long_bf16", GDN, 1, 65536, 16, 128, 128, 16, 64, "bf16",
                            "softplus16", True, 0.0, 105),
}
DO_SEED = 104          # upstream gradient of the GDN backward workload
DECODE_SEED = 106      # decode: N=256 sequences, H=16, E=16, K=V=128


def _torch_dtype(dtype: str):
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def _unit(rng, shape, nonneg=False):
    x = rng.standard_normal(shape)
    if nonneg:
        x = np.logaddexp(0.0, x)        # softplus, as the second-key activation
    n = np.linalg.norm(x, axis=-1, keepdims=True)
    return x / np.maximum(n, 1e-30)


def _gates(rng, shape, recipe):
    x = rng.standard_normal(shape)
    if recipe == "logsigmoid_n3":       # a = sigmoid(x), x ~ N(3, 1)
        return -np.logaddexp(0.0, -(x + 3.0))
    if recipe == "softplus16":          # log a = -softplus(x) / 16, x ~ N(0, 1)
        return -np.logaddexp(0.0, x) / 16.0
    raise ValueError(recipe)


def make_inputs(cfg: Config, B: Optional[int] = None, T: Optional[int] = None,
                H: Optional[int] = None, seed: Optional[int] = None,
                nonneg_second: bool = False, gate_scale: float = 1.0):
    """Returns a dict of CPU torch tensors: q, k, v, q2, k2 in the config dtype,
    g, beta (or None), s0 (or None) in float32."""
    B = cfg.B if B is None else B
    T = cfg.T if T is None else T
    H = cfg.H if H is None else H
    rng = np.random.Generator(np.random.PCG64(cfg.seed if seed is None else seed))
    dt = _torch_dtype(cfg.dtype)
    K, V, E = cfg.K, cfg.V, cfg.E
    out = {}
    out["q"] = torch.from_numpy(_unit(rng, (B, T, H, K))).to(dt)
    out["k"] = torch.from_numpy(_unit(rng, (B, T, H, K))).to(dt)
    out["v"] = torch.from_numpy(rng.standard_normal((B, T, H, V))).to(dt)
    out["q2"] = torch.from_numpy(_unit(rng, (B, T, H, E), nonneg_second)).to(dt)
    out["k2"] = torch.from_numpy(_unit(rng, (B, T, H, E), nonneg_second)).to(dt)
    out["g"] = torch.from_numpy(gate_scale * _gates(rng, (B, T, H, E), cfg.gate)).float()
    if cfg.beta or cfg.variant == GDN:
        out["beta"] = torch.from_numpy(1.0 / (1.0 + np.exp(-rng.standard_normal((B, T, H))))).float()
    else:
        out["beta"] = None
    if cfg.s0_std > 0:
        out["s0"] = torch.from_numpy(cfg.s0_std * rng.standard_normal((B, H, E, K, V))).float()
    else:
        out["s0"] = None
    return out


def make_dO(cfg: Config, B=None, T=None, H=None, seed=DO_SEED):
    B = cfg.B if B is None else B
    T = cfg.T if T is None else T
    H = cfg.H if H is None else H
    rng = np.random.Generator(np.random.PCG64(seed))
    return torch.from_numpy(rng.standard_normal((B, T, H, cfg.V))).to(_torch_dtype(cfg.dtype))


def make_decode_state(N, H, E, K, V, std=0.02, seed=DECODE_SEED):
    rng = np.random.Generator(np.random.PCG64(seed))
    return torch.from_numpy(std * rng.standard_normal((N, H, E, K, V), dtype=np.float32))


def make_decode_token(N, H, K, V, E, dtype="bf16", seed=DECODE_SEED + 1,
                      variant=GDN):
    """One fresh token per (n, h) with the distributions above."""
    rng = np.random.Generator(np.random.PCG64(seed))
    dt = _torch_dtype(dtype)
    out = {
        "q": torch.from_numpy(_unit(rng, (N, H, K))).to(dt),
        "k": torch.from_numpy(_unit(rng, (N, H, K))).to(dt),
        "v": torch.from_numpy(rng.standard_normal((N, H, V))).to(dt),
        "q2": torch.from_numpy(_unit(rng, (N, H, E))).to(dt),
        "k2": torch.from_numpy(_unit(rng, (N, H, E))).to(dt),
        "g": torch.from_numpy(_gates(rng, (N, H, E), "softplus16")).float(),
    }
    b = torch.from_numpy(1.0 / (1.0 + np.exp(-rng.standard_normal((N, H))))).float()
    out["beta"] = b if variant == GDN else None
    return out


def to64(x):
    """The cast values as float64 numpy (what the oracle consumes)."""
    if x is None:
        return None
    return x.detach().to("cpu", torch.float64).numpy()

"""Plants plausible mistakes in a private copy of the C oracle (on the CPU) and
checks that the pins catch each one: a sign flip, a dropped term, a wrong
index and a swapped operand in the forward, and in the backward."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
from oracle import forms

SGLA, GDN = oracle.SGLA, oracle.GDN
SRC = os.path.join(os.path.dirname(oracle.__file__), "tla_oracle.c")

FWD_MUTANTS = {
    "erase_sign": ("beta * (v[j] - r[j]) : beta * v[j]", "beta * (v[j] + r[j]) : beta * v[j]"),
    "no_decay": ("for (size_t i = 0; i < KV; ++i) Se[i] *= a;", "for (size_t i = 0; i < KV; ++i) Se[i] *= 1.0;"),
    "query_uses_key2": ("const double rho = q2[e] * q[kk];\n      const double* row = S + e * KV + (size_t)kk * V;\n      for (int j = 0; j < V; ++j) o[j]",
                        "const double rho = k2[e] * q[kk];\n      const double* row = S + e * KV + (size_t)kk * V;\n      for (int j = 0; j < V; ++j) o[j]"),
    "sgla_drops_beta": ("beta * (v[j] - r[j]) : beta * v[j]", "beta * (v[j] - r[j]) : v[j]"),
    "retrieval_wrong_key": ("const double kap = k2[e] * k[kk];\n        const double* row = S + e * KV",
                            "const double kap = k2[e] * q[kk];\n        const double* row = S + e * KV"),
    "read_before_write": ("  /* read with the joint query q2 (x) q */\n  for (int j = 0; j < V; ++j) o[j] = 0.0;",
                          "  /* read with the joint query q2 (x) q */\n  for (int j = 0; j < V; ++j) o[j] = 0.0;\n  for (int e = 0; e < E; ++e) for (int kk = 0; kk < K; ++kk) { double* row = S + e * KV + (size_t)kk * V; for (int j = 0; j < V; ++j) row[j] -= k2[e] * k[kk] * w[j]; }"),
}
BWD_MUTANTS = {
    "dg_missing": ("dgt[e] = acc;", "dgt[e] = 0.0 * acc;"),
    "dr_sign": ("dr[j] = -bt * dw[j];", "dr[j] = bt * dw[j];"),
    "dS_not_decayed": ("            drow[i] *= a;\n", "            drow[i] *= 1.0;\n"),
    "dq2_wrong_factor": ("for (int kk = 0; kk < K; ++kk) acc += qt[kk] * drho[e * K + kk];",
                         "for (int kk = 0; kk < K; ++kk) acc += kt[kk] * drho[e * K + kk];"),
    "dbeta_gdn_drops_r": ("db += dw[j] * (vt[j] - r[j]);", "db += dw[j] * vt[j];"),
}


def build_mutant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) >= 1, name
    mut = src.replace(old, new, 1)
    if name == "read_before_write":
        # the inserted loop undoes the write before the read and must be
        # re-applied after it: add the write back once the read is done
        mut = mut.replace(
            "      for (int j = 0; j < V; ++j) o[j] += rho * row[j];\n    }\n}",
            "      for (int j = 0; j < V; ++j) o[j] += rho * row[j];\n    }\n"
            "  for (int e = 0; e < E; ++e) for (int kk = 0; kk < K; ++kk) { double* row = S + e * KV + (size_t)kk * V; for (int j = 0; j < V; ++j) row[j] += k2[e] * k[kk] * w[j]; }\n}", 1)
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(mut)
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-std=c99", "-o", str(so), str(c), "-lm"],
                   check=True)
    lib = ctypes.CDLL(str(so))
    P, I = ctypes.c_void_p, ctypes.c_int
    lib.oracle_fwd.argtypes = [I] * 7 + [P] * 10
    lib.oracle_bwd.argtypes = [I] * 7 + [P] * 18
    return lib


def ptr(x):
    return None if x is None else x.ctypes.data_as(ctypes.c_void_p)


def mut_fwd(lib, variant, d):
    B, T, H, K = d["q"].shape
    V, E = d["v"].shape[-1], d["q2"].shape[-1]
    o = np.zeros((B, T, H, V)); sf = np.zeros((B, H, E, K, V))
    rc = lib.oracle_fwd(variant, B, T, H, K, V, E, *[ptr(d[n]) for n in
                        ("q", "k", "v", "q2", "k2", "g", "beta", "s0")], ptr(o), ptr(sf))
    assert rc == 0
    return o, sf


def mut_bwd(lib, variant, d, dO, dSf):
    B, T, H, K = d["q"].shape
    V, E = d["v"].shape[-1], d["q2"].shape[-1]
    out = [np.zeros((B, T, H, K)), np.zeros((B, T, H, K)), np.zeros((B, T, H, V)),
           np.zeros((B, T, H, E)), np.zeros((B, T, H, E)), np.zeros((B, T, H, E)),
           np.zeros((B, T, H)), np.zeros((B, H, E, K, V))]
    rc = lib.oracle_bwd(variant, B, T, H, K, V, E, *[ptr(d[n]) for n in
                        ("q", "k", "v", "q2", "k2", "g", "beta", "s0")], ptr(dO), ptr(dSf),
                        *[ptr(x) for x in out])
    assert rc == 0
    return out


def inputs(seed, T=10):
    rng = np.random.default_rng(seed)
    B, H, K, V, E = 1, 2, 3, 2, 3
    unit = lambda s: (lambda x: x / np.linalg.norm(x, axis=-1, keepdims=True))(rng.standard_normal(s))
    return dict(q=unit((B, T, H, K)), k=unit((B, T, H, K)), v=rng.standard_normal((B, T, H, V)),
                q2=unit((B, T, H, E)), k2=unit((B, T, H, E)), g=rng.uniform(-0.6, -0.01, (B, T, H, E)),
                beta=rng.uniform(0.1, 0.9, (B, T, H)), s0=0.5 * rng.standard_normal((B, H, E, K, V)))


@pytest.mark.parametrize("name", sorted(FWD_MUTANTS))
def test_forward_mutant_is_caught(tmp_path, name):
    lib = build_mutant(tmp_path, name, *FWD_MUTANTS[name])
    d = inputs(50)
    caught = []
    for variant in (SGLA, GDN):
        o, sf = mut_fwd(lib, variant, d)
        o2, sf2 = forms.flat_joint_key(variant, **d)
        caught.append(not np.allclose(o, o2, rtol=0, atol=1e-9))
    o = mut_fwd(lib, SGLA, d)[0]
    caught.append(not np.allclose(o, forms.quadratic_sgla(**d), rtol=0, atol=1e-9))
    assert any(caught), f"mutant {name} passed every forward pin"


@pytest.mark.parametrize("name", sorted(BWD_MUTANTS))
def test_backward_mutant_is_caught(tmp_path, name):
    lib = build_mutant(tmp_path, name, *BWD_MUTANTS[name])
    d = inputs(51, T=6)
    rng = np.random.default_rng(52)
    dO = rng.standard_normal(d["v"].shape)
    dSf = rng.standard_normal(d["s0"].shape)
    names = ("q", "k", "v", "q2", "k2", "g", "beta", "s0")
    grads = mut_bwd(lib, GDN, d, dO, dSf)

    def L(dd):
        o, sf = oracle.fwd(GDN, *[dd[n] for n in names])
        return float(np.sum(o * dO) + np.sum(sf * dSf))

    h = 1e-6
    bad = False
    for n, gmut in zip(names, grads):
        x = d[n]
        for i in np.ndindex(x.shape):
            old = x[i]
            x[i] = old + h; lp = L(d)
            x[i] = old - h; lm = L(d)
            x[i] = old
            if abs((lp - lm) / (2 * h) - gmut[i]) > 1e-5:
                bad = True
                break
        if bad:
            break
    assert bad, f"mutant {name} passed the finite-difference pin"

"""GPU parity of the mixer's output side (RMSNorm times a sigmoid gate, the
last line of the mixer in Alg. 2): tla_out_gate_fwd / tla_out_gate_bwd
against the fp64 oracle, max|err| / RMS(ref) per tensor.

Tolerance (fp32 outputs and dw, both dtypes): 1e-5, the operator's fp32
bar.  Each output element is a chain of about ten fp32 roundings (2^-24
each) after the row's mean square, a sum of V <= 256 squares reduced over
a lane group (log2 V + 1 roundings); with Gaussian inputs max|ref| is a few
RMS(ref), so the expected max|err| / RMS(ref) is a few 1e-6 (measured at
most 4e-6 over these cases).  dw sums the rows in a fixed order (a
workgroup's lanes, then the workgroups), each term exact to about ten
roundings: the same few 1e-6 relative to RMS(dw) at these row counts."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36529_amd as tla
from helpers import rel_err

pytestmark = pytest.mark.gpu
TOL_F32 = 1e-5  # max|err| / RMS(ref), fp32 outputs and dw


def within_bf16_rounding(got, ref):
    """bf16 outputs are one rounding of an fp32 result (at most 2^-9 relative):
    elementwise |got - ref| <= 2^-8 |ref| + 1e-5 RMS(ref)."""
    rms = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    return bool(np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-5 * rms))


def make(rows, V, dtype, seed, scale=1.0):
    g = torch.Generator().manual_seed(seed)
    o = (scale * torch.randn(rows, V, generator=g)).to(dtype)
    z = (2.0 * torch.randn(rows, V, generator=g)).to(dtype)
    w = (1.0 + 0.5 * torch.randn(V, generator=g)).float()
    dy = torch.randn(rows, V, generator=g).to(dtype)
    return o, z, w, dy


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def check(rows, V, dtype, seed=0, eps=1e-6, scale=1.0):
    o, z, w, dy = make(rows, V, dtype, seed, scale)
    od, zd, wd, dyd = (t.cuda() for t in (o, z, w, dy))
    y = tla.out_gate_fwd(od, zd, wd, eps)
    do, dz, dw = tla.out_gate_bwd(od, zd, wd, dyd, eps)
    torch.cuda.synchronize()
    ry = oracle.out_gate_fwd(f64(o), f64(z), f64(w), eps)
    rdo, rdz, rdw = oracle.out_gate_bwd(f64(o), f64(z), f64(w), eps, f64(dy))
    errs = {"y": rel_err(f64(y), ry), "do": rel_err(f64(do), rdo), "dz": rel_err(f64(dz), rdz),
            "dw": rel_err(f64(dw), rdw)}
    print(f"rows={rows} V={V} {dtype}: " + " ".join(f"{k}={v:.1e}" for k, v in errs.items()), flush=True)
    # dw sums the rows in fp32 from the same (exact) inputs: fp32 accuracy for both dtypes
    assert errs["dw"] <= TOL_F32, errs
    if dtype == torch.float32:
        bad = {k: v for k, v in errs.items() if v > TOL_F32}
        assert not bad, bad
    else:
        for k, got, ref in (("y", y, ry), ("do", do, rdo), ("dz", dz, rdz)):
            assert within_bf16_rounding(f64(got), ref), k


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("V", [16, 32, 64, 128, 256])
@pytest.mark.parametrize("rows", [1, 37, 1000])
def test_parity(rows, V, dtype):
    check(rows, V, dtype, seed=rows + V)


def test_scaled_and_zero_rows():
    check(300, 128, torch.float32, seed=5, scale=1e-3, eps=1e-6)
    o, z, w, dy = make(64, 128, torch.float32, 6)
    o[3] = 0.0
    y = tla.out_gate_fwd(o.cuda(), z.cuda(), w.cuda(), 1e-6)
    do, dz, dw = tla.out_gate_bwd(o.cuda(), z.cuda(), w.cuda(), dy.cuda(), 1e-6)
    torch.cuda.synchronize()
    assert torch.all(y[3] == 0) and torch.isfinite(do).all() and torch.isfinite(dw).all()


def test_empty():
    o = torch.empty(0, 128, device="cuda")
    w = torch.ones(128, device="cuda")
    y = tla.out_gate_fwd(o, o, w)
    do, dz, dw = tla.out_gate_bwd(o, o, w, o)
    torch.cuda.synchronize()
    assert y.numel() == 0 and torch.equal(dw.cpu(), torch.zeros(128))


def test_metric_shape_sampled_rows_and_determinism():
    """B4 T4096 H8 V128 bf16 (the output of the forward at the bench shape):
    sampled rows against the oracle; dw against the oracle's full sum; two
    backward calls bitwise equal."""
    B, T, H, V = 4, 4096, 8, 128
    o, z, w, dy = make(B * T * H, V, torch.bfloat16, 11)
    od, zd, wd, dyd = (t.cuda() for t in (o, z, w, dy))
    y = tla.out_gate_fwd(od.view(B, T, H, V), zd.view(B, T, H, V), wd)
    do, dz, dw = tla.out_gate_bwd(od, zd, wd, dyd)
    do2, dz2, dw2 = tla.out_gate_bwd(od, zd, wd, dyd)
    torch.cuda.synchronize()
    assert torch.equal(dw, dw2) and torch.equal(do, do2) and torch.equal(dz, dz2)
    rows = np.random.default_rng(0).choice(B * T * H, 512, replace=False)
    ry = oracle.out_gate_fwd(f64(o[rows]), f64(z[rows]), f64(w), 1e-6)
    rdo, rdz, _ = oracle.out_gate_bwd(f64(o[rows]), f64(z[rows]), f64(w), 1e-6, f64(dy[rows]))
    assert within_bf16_rounding(f64(y.view(-1, V)[rows]), ry)
    assert within_bf16_rounding(f64(do[rows]), rdo)
    assert within_bf16_rounding(f64(dz[rows]), rdz)
    _, _, rdw = oracle.out_gate_bwd(f64(o), f64(z), f64(w), 1e-6, f64(dy))
    assert rel_err(f64(dw), rdw) < 1e-4

"""GPU parity of the mixer's input side after the projection GEMM (causal
depthwise convolution, SiLU on q, k, v, softplus on q', k', L2 normalisation
of q, k, q', k'; section "Input projections", Alg. 2): tla_conv_in_fwd /
tla_conv_in_bwd against the fp64 oracle.

Tolerances.  fp32 outputs and the tap gradient dw (fp32 for both dtypes):
max|err| / RMS(ref) <= 1e-5 per tensor, the operator's fp32 bar.  A value
is a W-tap sum, an activation and a division by the norm of its K or E
entries (a sum of at most 128 squares, log2 128 + 1 roundings): a few tens
of fp32 roundings at most, so the error is a few 1e-6 of RMS(ref)
(measured at most 3.4e-6, including inputs scaled by 1e4 and eps = 0).  dw
sums tokens in a fixed order, a few hundred products per partial and then
the partials pairwise; at the full shape (16384 tokens) its measured error
is 1.3e-6 of RMS(dw).  bf16 outputs are one rounding of an fp32 result:
elementwise |err| <= 2^-8 |ref| + 1e-5 RMS(ref)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36529_amd as tla
from helpers import rel_err

pytestmark = pytest.mark.gpu
TOL = 1e-5
NAMES = ("q", "k", "v", "q2", "k2")


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def within_bf16_rounding(got, ref):
    rms = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    return bool(np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-5 * rms))


def make(B, T, H, K, V, E, W, dtype, seed):
    """y ~ N(0, 1) (projection outputs of a normalised input); taps
    U(-1/sqrt W, 1/sqrt W) (depthwise fan-in W); output gradients ~ N(0, 1)."""
    g = torch.Generator().manual_seed(seed)
    C = H * (2 * K + V + 2 * E)
    y = torch.randn(B, T, C, generator=g).to(dtype)
    w = ((torch.rand(W, C, generator=g) * 2 - 1) / W ** 0.5).float()
    grads = tuple(torch.randn(B, T, H, d, generator=g).to(dtype) for d in (K, K, V, E, E))
    return y, w, grads


def check(B, T, H, K, V, E, W, dtype, seed=0, eps=1e-6):
    y, w, grads = make(B, T, H, K, V, E, W, dtype, seed)
    yd, wd = y.cuda(), w.cuda()
    gd = tuple(t.cuda() for t in grads)
    outs = tla.conv_in_fwd(yd, wd, H, K, V, E, eps)
    dy, dw = tla.conv_in_bwd(yd, wd, H, K, V, E, gd, eps)
    torch.cuda.synchronize()
    ref = oracle.conv_in_fwd(f64(y), f64(w), H, K, V, E, eps)
    rdy, rdw = oracle.conv_in_bwd(f64(y), f64(w), H, K, V, E, eps, dict(zip(NAMES, (f64(t) for t in grads))))
    print(f"B={B} T={T} H={H} K={K} V={V} E={E} W={W} {dtype}", flush=True)
    pairs = [(n, f64(o), ref[n]) for n, o in zip(NAMES, outs)] + [("dy", f64(dy), rdy)]
    for n, got, r in pairs:
        if dtype == torch.float32:
            assert rel_err(got, r) <= TOL, (n, rel_err(got, r))
        else:
            assert within_bf16_rounding(got, r), n
    assert rel_err(f64(dw), rdw) <= TOL, ("dw", rel_err(f64(dw), rdw))


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("W", [1, 2, 3, 4])
def test_parity_taps(W, dtype):
    check(2, 45, 3, 16, 24, 8, W, dtype, seed=W)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("shape", [(1, 1, 1, 8, 8, 8), (1, 31, 2, 32, 16, 16), (2, 33, 4, 64, 64, 8),
                                   (1, 100, 8, 128, 128, 8), (3, 70, 2, 128, 40, 16),
                                   (1, 65, 2, 256, 256, 32)])
def test_parity_shapes(shape, dtype):
    B, T, H, K, V, E = shape
    check(B, T, H, K, V, E, 4, dtype, seed=sum(shape))


def test_eps_zero_and_large_inputs():
    check(2, 40, 2, 32, 16, 8, 4, torch.float32, seed=9, eps=0.0)
    y, w, grads = make(1, 50, 2, 32, 16, 8, 3, torch.float32, 10)
    y = y * 8.0  # pre-activations up to ~40: saturated sigmoid, softplus' linear branch
    outs = tla.conv_in_fwd(y.cuda(), w.cuda(), 2, 32, 16, 8, 1e-6)
    dy, dw = tla.conv_in_bwd(y.cuda(), w.cuda(), 2, 32, 16, 8, tuple(t.cuda() for t in grads), 1e-6)
    torch.cuda.synchronize()
    ref = oracle.conv_in_fwd(f64(y), f64(w), 2, 32, 16, 8, 1e-6)
    rdy, rdw = oracle.conv_in_bwd(f64(y), f64(w), 2, 32, 16, 8, 1e-6, dict(zip(NAMES, (f64(t) for t in grads))))
    for n, o in zip(NAMES, outs):
        assert rel_err(f64(o), ref[n]) <= TOL, n
    assert rel_err(f64(dy), rdy) <= TOL and rel_err(f64(dw), rdw) <= TOL


def test_empty():
    H, K, V, E, W = 2, 16, 16, 8, 4
    C = H * (2 * K + V + 2 * E)
    y = torch.empty(1, 0, C, device="cuda")
    w = torch.randn(W, C, device="cuda")
    outs = tla.conv_in_fwd(y, w, H, K, V, E)
    grads = tuple(torch.empty(1, 0, H, d, device="cuda") for d in (K, K, V, E, E))
    dy, dw = tla.conv_in_bwd(y, w, H, K, V, E, grads)
    torch.cuda.synchronize()
    assert all(o.numel() == 0 for o in outs) and dy.numel() == 0
    assert torch.equal(dw.cpu(), torch.zeros(W, C))


def test_metric_shape_windows_and_determinism():
    """B4 T4096 H8 K=V=128 E=8 W=4 bf16 (the operator's inputs at the bench
    shape): outputs and dy on sampled windows of tokens (the oracle run on the
    window plus its halo), dw against the oracle's full sum, two backward calls
    bitwise equal."""
    B, T, H, K, V, E, W = 4, 4096, 8, 128, 128, 8, 4
    y, w, grads = make(B, T, H, K, V, E, W, torch.bfloat16, 21)
    yd, wd = y.cuda(), w.cuda()
    gd = tuple(t.cuda() for t in grads)
    outs = tla.conv_in_fwd(yd, wd, H, K, V, E)
    dy, dw = tla.conv_in_bwd(yd, wd, H, K, V, E, gd)
    dy2, dw2 = tla.conv_in_bwd(yd, wd, H, K, V, E, gd)
    torch.cuda.synchronize()
    assert torch.equal(dy, dy2) and torch.equal(dw, dw2)
    rng = np.random.default_rng(2)
    for b, s in [(0, 0), (3, T - 32)] + [(int(rng.integers(B)), int(rng.integers(3, T - 35))) for _ in range(6)]:
        lo, hi = max(s - (W - 1), 0), min(s + 32 + (W - 1), T)
        ys = f64(y[b:b + 1, lo:hi])
        gs = {n: f64(g[b:b + 1, lo:hi]) for n, g in zip(NAMES, grads)}
        ref = oracle.conv_in_fwd(ys, f64(w), H, K, V, E, 1e-6)
        rdy, _ = oracle.conv_in_bwd(ys, f64(w), H, K, V, E, 1e-6, gs)
        a, e = s - lo, s - lo + min(32, T - s)
        for n, o in zip(NAMES, outs):
            assert within_bf16_rounding(f64(o[b, s:s + e - a]), ref[n][0, a:e]), (n, b, s)
        assert within_bf16_rounding(f64(dy[b, s:s + e - a]), rdy[0, a:e]), ("dy", b, s)
    _, rdw = oracle.conv_in_bwd(f64(y), f64(w), H, K, V, E, 1e-6, dict(zip(NAMES, (f64(g) for g in grads))))
    assert rel_err(f64(dw), rdw) <= TOL

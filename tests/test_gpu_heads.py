"""GPU parity of the mixer's gate heads (Alg. 2: the log forget gate
g = -exp(A) softplus(x + b) and the write strength beta = sigmoid(x_beta)):
tla_gate_heads_fwd / tla_gate_heads_bwd against the fp64 oracle.

Tolerances.  g, beta and the fp32 dx, dxb are a handful of fp32 operations on
exact inputs: elementwise relative error <= 1e-5.  bf16 dx, dxb are one
rounding of such a value (elementwise, see within_bf16_rounding).  dA, db sum
n tokens in fp32 (sequential runs of 64 tokens, then a tree over the runs):
the classic bound is about (64 + log2 runs) * 2^-24 * sum|terms| per column,
so |err| <= 1e-5 * sum over tokens of |term|."""
import numpy as np
import pytest
import torch

import oracle
import paper_2609_36529_amd as tla

pytestmark = pytest.mark.gpu
REL = 1e-5


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def within_bf16_rounding(got, ref):
    """One bf16 rounding of an fp32 result: |got - ref| <= 2^-8 |ref| + 1e-5 RMS(ref)."""
    rms = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    return bool(np.all(np.abs(got - ref) <= 2.0 ** -8 * np.abs(ref) + 1e-5 * rms))


def close_rel(got, ref, rel=REL):
    return bool(np.all(np.abs(got - ref) <= rel * np.abs(ref) + 1e-30))


def make(tokens, H, E, dtype, seed, with_beta=True, xscale=1.0):
    """A = log U(1, 16), b = softplus^-1(dt) with dt log-uniform in [1e-3, 0.1],
    pre-activations x, x_beta ~ N(0, xscale^2), upstream gradients ~ N(0, 1)."""
    g = torch.Generator().manual_seed(seed)
    x = (xscale * torch.randn(tokens, H, E, generator=g)).to(dtype)
    xb = (xscale * torch.randn(tokens, H, generator=g)).to(dtype) if with_beta else None
    A = torch.log(1.0 + 15.0 * torch.rand(H, E, generator=g)).float()
    dt = torch.exp(np.log(1e-3) + (np.log(0.1) - np.log(1e-3)) * torch.rand(H, E, generator=g, dtype=torch.float64))
    b = torch.log(torch.expm1(dt)).float()
    dg = torch.randn(tokens, H, E, generator=g).float()
    dbeta = torch.randn(tokens, H, generator=g).float() if with_beta else None
    return x, xb, A, b, dg, dbeta


def cuda(t):
    return None if t is None else t.cuda()


def check(tokens, H, E, dtype, seed=0, with_beta=True, xscale=1.0):
    x, xb, A, b, dg, dbeta = make(tokens, H, E, dtype, seed, with_beta, xscale)
    xd, xbd, Ad, bd, dgd, dbd = (cuda(t) for t in (x, xb, A, b, dg, dbeta))
    g, beta = tla.gate_heads_fwd(xd, xbd, Ad, bd)
    dx, dxb, dA, db = tla.gate_heads_bwd(xd, xbd, Ad, bd, dgd, dbd)
    torch.cuda.synchronize()
    xb64 = f64(xb) if with_beta else np.zeros((tokens, H))
    dbeta64 = f64(dbeta) if with_beta else np.zeros((tokens, H))
    rg, rbeta = oracle.gate_heads_fwd(f64(x), xb64, f64(A), f64(b))
    rdx, rdxb, rdA, rdb = oracle.gate_heads_bwd(f64(x), xb64, f64(A), f64(b), f64(dg), dbeta64)
    print(f"tokens={tokens} H={H} E={E} {dtype} beta={with_beta} xscale={xscale}", flush=True)
    assert close_rel(f64(g), rg), "g"
    if dtype == torch.float32:
        assert close_rel(f64(dx), rdx), "dx"
    else:
        assert within_bf16_rounding(f64(dx), rdx), "dx"
    if with_beta:
        assert close_rel(f64(beta), rbeta), "beta"
        if dtype == torch.float32:
            assert close_rel(f64(dxb), rdxb), "dxb"
        else:
            assert within_bf16_rounding(f64(dxb), rdxb), "dxb"
    else:
        assert beta is None and dxb is None
    # summation bound per column
    absA = np.abs(f64(dg) * rg).reshape(-1, H, E).sum(axis=0)
    absb = np.abs(rdx).reshape(-1, H, E).sum(axis=0)
    assert np.all(np.abs(f64(dA) - rdA) <= 1e-5 * absA + 1e-30), "dA"
    assert np.all(np.abs(f64(db) - rdb) <= 1e-5 * absb + 1e-30), "db"


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("HE", [(8, 1), (8, 8), (3, 5), (16, 32)])
@pytest.mark.parametrize("tokens", [1, 63, 64, 65, 1000])
def test_parity(tokens, HE, dtype):
    H, E = HE
    check(tokens, H, E, dtype, seed=tokens * 31 + H * E)


def test_without_beta_and_many_columns():
    """sGLA (no write strength) and more columns than threads per workgroup."""
    check(200, 8, 4, torch.bfloat16, seed=3, with_beta=False)
    check(130, 64, 9, torch.float32, seed=4)


def test_large_pre_activations():
    """|x + b| up to about 60 (x ~ N(0, 12^2)): both sides of softplus'
    large-argument branch and a saturated sigmoid, while exp(-|x + b|) stays a
    normal fp32 number, so relative accuracy is still owed."""
    check(500, 4, 8, torch.float32, seed=5, xscale=12.0)


def test_empty():
    H, E = 8, 8
    x = torch.empty(0, H, E, device="cuda")
    xb = torch.empty(0, H, device="cuda")
    A = torch.zeros(H, E, device="cuda")
    b = torch.zeros(H, E, device="cuda")
    g, beta = tla.gate_heads_fwd(x, xb, A, b)
    dx, dxb, dA, db = tla.gate_heads_bwd(x, xb, A, b, x, xb)
    torch.cuda.synchronize()
    assert g.numel() == 0 and beta.numel() == 0
    assert torch.equal(dA.cpu(), torch.zeros(H, E)) and torch.equal(db.cpu(), torch.zeros(H, E))


def test_metric_shape_sampled_and_determinism():
    """B4 T4096 H8 E8 bf16 pre-activations (the gates of the bench shape):
    sampled tokens against the oracle, dA / db against the oracle's full sum,
    two backward calls bitwise equal."""
    B, T, H, E = 4, 4096, 8, 8
    n = B * T
    x, xb, A, b, dg, dbeta = make(n, H, E, torch.bfloat16, 12)
    xd, xbd, Ad, bd, dgd, dbd = (cuda(t) for t in (x, xb, A, b, dg, dbeta))
    g, beta = tla.gate_heads_fwd(xd.view(B, T, H, E), xbd.view(B, T, H), Ad, bd)
    dx, dxb, dA, db = tla.gate_heads_bwd(xd, xbd, Ad, bd, dgd, dbd)
    dx2, dxb2, dA2, db2 = tla.gate_heads_bwd(xd, xbd, Ad, bd, dgd, dbd)
    torch.cuda.synchronize()
    assert torch.equal(dA, dA2) and torch.equal(db, db2) and torch.equal(dx, dx2) and torch.equal(dxb, dxb2)
    rows = np.random.default_rng(1).choice(n, 512, replace=False)
    rg, rbeta = oracle.gate_heads_fwd(f64(x[rows]), f64(xb[rows]), f64(A), f64(b))
    rdx, rdxb, _, _ = oracle.gate_heads_bwd(f64(x[rows]), f64(xb[rows]), f64(A), f64(b), f64(dg[rows]),
                                             f64(dbeta[rows]))
    assert close_rel(f64(g.view(n, H, E)[rows]), rg)
    assert close_rel(f64(beta.view(n, H)[rows]), rbeta)
    assert within_bf16_rounding(f64(dx[rows]), rdx)
    assert within_bf16_rounding(f64(dxb[rows]), rdxb)
    rg_all, _ = oracle.gate_heads_fwd(f64(x), f64(xb), f64(A), f64(b))
    rdx_all, _, rdA, rdb = oracle.gate_heads_bwd(f64(x), f64(xb), f64(A), f64(b), f64(dg), f64(dbeta))
    absA = np.abs(f64(dg) * rg_all).sum(axis=0)
    absb = np.abs(rdx_all).sum(axis=0)
    assert np.all(np.abs(f64(dA) - rdA) <= 1e-5 * absA)
    assert np.all(np.abs(f64(db) - rdb) <= 1e-5 * absb)

"""Pins of the fp64 input-projection reference (one GEMM over all channel
blocks, then the convolution, activations and normalisations; section
"Input projections" and Alg. 2): the GEMM against an explicit triple loop,
the whole forward against the hand-worked values of the input side through
a scaled identity projection, causality through the projection, and the
backward against central finite differences on every input."""
import math

import numpy as np

import oracle.proj_in as pi


def test_projection_is_the_explicit_sum():
    """y[b, t, c] = sum_d u[b, t, d] Wp[c, d], written as loops; Dm != Ctot
    and a non-symmetric square case, so a transposed operand fails."""
    rng = np.random.default_rng(11)
    for B, T, Dm, C in ((2, 3, 5, 7), (1, 4, 6, 6)):
        u = rng.standard_normal((B, T, Dm))
        Wp = rng.standard_normal((C, Dm))
        y = pi.project(u, Wp)
        ref = np.zeros((B, T, C))
        for b in range(B):
            for t in range(T):
                for c in range(C):
                    s = 0.0
                    for d in range(Dm):
                        s += u[b, t, d] * Wp[c, d]
                    ref[b, t, c] = s
        np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


def test_worked_example_through_a_scaled_identity():
    """Wp = 2 I (Dm = Ctot = 9) and u = y / 2 reproduce the input side's
    hand-worked example (H = 1, K = 2, V = 1, E = 2, W = 2, taps (0.5, 1),
    eps = 0): q = (3, -1) / sqrt 10 at both tokens, k = (-1, 3) / sqrt 10 at
    token 0, v = (3/4) ln 3 at token 0 and (ln 3 / 2) sqrt 3 / (1 + sqrt 3)
    at token 1, q' = (1, 1) / sqrt 2, k' = (ln 2, 1) / sqrt(ln^2 2 + 1)."""
    l3, le = math.log(3.0), math.log(math.e - 1.0)
    y = np.zeros((1, 2, 9))
    y[0, 0] = [l3, -l3, -l3, l3, l3, le, le, 0.0, le]
    y[0, 1] = [l3 / 2, -l3 / 2, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0, 0.0]
    w = np.stack([np.full(9, 0.5), np.ones(9)])
    o, yy = pi.proj_in_fwd(y / 2, 2.0 * np.eye(9), w, 1, 2, 1, 2, 0.0)
    np.testing.assert_allclose(yy, y, rtol=1e-15, atol=0)
    s10, r3 = math.sqrt(10.0), math.sqrt(3.0)
    np.testing.assert_allclose(o["q"][0, :, 0], [[3 / s10, -1 / s10]] * 2, rtol=1e-14)
    np.testing.assert_allclose(o["k"][0, 0, 0], [-1 / s10, 3 / s10], rtol=1e-14)
    np.testing.assert_allclose(o["v"][0, :, 0, 0], [0.75 * l3, l3 / 2 * r3 / (1 + r3)], rtol=1e-14)
    np.testing.assert_allclose(o["q2"][0, 0, 0], [1 / math.sqrt(2.0)] * 2, rtol=1e-14)
    n = math.sqrt(math.log(2.0) ** 2 + 1.0)
    np.testing.assert_allclose(o["k2"][0, 0, 0], [math.log(2.0) / n, 1 / n], rtol=1e-14)


def test_permuted_projection_rows_permute_channels_of_the_same_block():
    """Swapping two rows of Wp inside the v block swaps those v channels and
    leaves every other output as it was (v is not normalised, so its channels
    do not mix)."""
    rng = np.random.default_rng(12)
    H, K, V, E, W, Dm = 1, 4, 6, 2, 3, 5
    C = H * (2 * K + V + 2 * E)
    u = rng.standard_normal((1, 6, Dm))
    Wp = rng.standard_normal((C, Dm))
    w = np.ones((W, C))  # the same taps on every channel
    a, _ = pi.proj_in_fwd(u, Wp, w, H, K, V, E, 1e-6)
    Wq = Wp.copy()
    i, j = 2 * K + 1, 2 * K + 4
    Wq[[i, j]] = Wq[[j, i]]
    b, _ = pi.proj_in_fwd(u, Wq, w, H, K, V, E, 1e-6)
    for name in ("q", "k", "q2", "k2"):
        np.testing.assert_array_equal(a[name], b[name])
    np.testing.assert_array_equal(a["v"][..., [1, 4]], b["v"][..., [4, 1]])
    np.testing.assert_array_equal(a["v"][..., [0, 2, 3, 5]], b["v"][..., [0, 2, 3, 5]])


def test_causal_through_the_projection():
    rng = np.random.default_rng(13)
    H, K, V, E, W, Dm = 2, 4, 3, 2, 4, 6
    C = H * (2 * K + V + 2 * E)
    u = rng.standard_normal((2, 10, Dm))
    Wp = rng.standard_normal((C, Dm))
    w = rng.standard_normal((W, C))
    base, _ = pi.proj_in_fwd(u, Wp, w, H, K, V, E, 1e-6)
    u2 = u.copy()
    u2[0, 5] += 0.5
    pert, _ = pi.proj_in_fwd(u2, Wp, w, H, K, V, E, 1e-6)
    for name in base:
        d = np.abs(pert[name] - base[name]).reshape(2, 10, -1).max(axis=-1)
        assert np.all(d[1] == 0) and np.all(d[0, :5] == 0) and np.all(d[0, 5 + W:] == 0), name
        assert np.all(d[0, 5:5 + W] > 0), name


def _loss(u, Wp, w, H, K, V, E, eps, g):
    o, _ = pi.proj_in_fwd(u, Wp, w, H, K, V, E, eps)
    return sum(float(np.sum(g[n] * o[n])) for n in g)


def test_backward_matches_finite_differences():
    rng = np.random.default_rng(14)
    H, K, V, E, W, Dm, B, T, eps = 1, 4, 4, 2, 3, 5, 2, 5, 1e-3
    C = H * (2 * K + V + 2 * E)
    u = rng.standard_normal((B, T, Dm))
    Wp = rng.standard_normal((C, Dm)) / math.sqrt(Dm)
    w = rng.standard_normal((W, C))
    shapes = {"q": K, "k": K, "v": V, "q2": E, "k2": E}
    g = {n: rng.standard_normal((B, T, H, s)) for n, s in shapes.items()}
    du, dWp, dw = pi.proj_in_bwd(u, Wp, w, H, K, V, E, eps, g)
    h = 1e-6

    def fd(arr, idx):
        old = arr[idx]
        arr[idx] = old + h
        lp = _loss(u, Wp, w, H, K, V, E, eps, g)
        arr[idx] = old - h
        lm = _loss(u, Wp, w, H, K, V, E, eps, g)
        arr[idx] = old
        return (lp - lm) / (2 * h)

    for arr, grad in ((u, du), (Wp, dWp), (w, dw)):
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            num[idx] = fd(arr, idx)
        np.testing.assert_allclose(grad, num, rtol=1e-6, atol=1e-8)


def _bf16(x):
    """Round to the nearest bf16 (ties to even), as fp64."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).float().to(torch.bfloat16).double().numpy()


def test_bf16_storage_alone_reaches_the_gradient_bounds_level():
    """The error level that bf16 storage alone causes in the projection's
    gradients: keep y in bf16, round dy to bf16 before the GEMMs and write du
    in bf16, with every operation otherwise exact (fp64).  This is what the
    GPU tests' bounds for du, dWp and dw must admit: relative l2 well below
    1e-2 and max|err| / RMS(ref) near 2e-2, under 4e-2."""
    import oracle.conv_in as oci
    rng = np.random.default_rng(15)
    B, T, Dm, H, K, V, E, W, eps = 1, 512, 256, 8, 128, 128, 8, 4, 1e-6
    C = H * (2 * K + V + 2 * E)
    u = _bf16(rng.standard_normal((B, T, Dm)))
    Wp = _bf16(rng.standard_normal((C, Dm)) / math.sqrt(Dm))
    w = (rng.random((W, C)) * 2 - 1) / math.sqrt(W)
    g = {n: _bf16(rng.standard_normal((B, T, H, d))) for n, d in
         (("q", K), ("k", K), ("v", V), ("q2", E), ("k2", E))}
    du, dWp, dw = pi.proj_in_bwd(u, Wp, w, H, K, V, E, eps, g)
    y16 = _bf16(pi.project(u, Wp))
    dy, dw16 = oci.conv_in_bwd(y16, w, H, K, V, E, eps, g)
    dy = _bf16(dy)
    du16 = _bf16(np.matmul(dy, Wp))
    dWp16 = np.matmul(dy.reshape(B * T, C).T, u.reshape(B * T, Dm))
    for got, ref in ((du16, du), (dWp16, dWp), (dw16, dw)):
        rms = np.sqrt(np.mean(ref * ref))
        mx = np.max(np.abs(got - ref)) / rms
        l2 = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        assert l2 < 5e-3 and 5e-3 < mx < 4e-2, (l2, mx)

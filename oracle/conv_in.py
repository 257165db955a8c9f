"""fp64 reference of the mixer's input side after the projection GEMM --
TEST INFRASTRUCTURE ONLY (tests, smoke and the bench's CPU baseline use it;
the HIP path never does).

Section "Input projections" and Alg. 2: one GEMM yields, per token, the
channels of q, k, v, q' and k' of every head; one causal depthwise
convolution runs over all of them; SiLU follows on the q, k and v channels
and softplus on the q' and k' channels; then q, k, q', k' are each divided
by their Euclidean norm (per token and head), v is not.

Layout of the GEMM output y: [B][T][Ctot] with Ctot = H (2K + V + 2E) and
channel blocks in the order q | k | v | q' | k', each head-major ([H][K],
[H][K], [H][V], [H][E], [H][E]).  Convolution taps w: [W][Ctot]; the output
at token t reads tokens t - W + 1 .. t of its own batch row (earlier tokens
count as zero), tap j weighting token t - (W - 1) + j.  Readings where the
paper is silent: no convolution bias, width W from the caller, and the norm
taken as x / sqrt(sum x^2 + eps) with eps from the caller (eps = 0 is the
plain definition).

Plain numpy; the backward is the chain rule written out.
"""
import numpy as np


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def _softplus(x):
    return np.logaddexp(0.0, x)


def _blocks(H, K, V, E):
    """(name, width per head, activation, normalised) in channel order."""
    return [("q", K, "silu", True), ("k", K, "silu", True), ("v", V, "silu", False),
            ("q2", E, "softplus", True), ("k2", E, "softplus", True)]


def causal_conv(y, w):
    """z[b, t, c] = sum_j w[j, c] y[b, t - (W - 1) + j, c], zero before t = 0."""
    y = np.asarray(y, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    W = w.shape[0]
    B, T, C = y.shape
    z = np.zeros_like(y)
    for j in range(W):
        shift = W - 1 - j  # tap j looks this many tokens back
        if shift < T:
            z[:, shift:, :] += w[j] * y[:, :T - shift, :]
    return z


def conv_in_fwd(y, w, H, K, V, E, eps):
    """-> dict q [B,T,H,K], k, v [B,T,H,V], q2 [B,T,H,E], k2 (fp64)."""
    z = causal_conv(y, w)
    B, T, _ = z.shape
    out, c0 = {}, 0
    for name, width, act, norm in _blocks(H, K, V, E):
        zb = z[:, :, c0:c0 + H * width].reshape(B, T, H, width)
        a = zb * _sigmoid(zb) if act == "silu" else _softplus(zb)
        if norm:
            a = a / np.sqrt(np.sum(a * a, axis=-1, keepdims=True) + eps)
        out[name] = a
        c0 += H * width
    return out


def conv_in_bwd(y, w, H, K, V, E, eps, grads):
    """Gradients (dy [B,T,Ctot], dw [W,Ctot]) of sum over the five outputs of
    <grads[name], output>; grads maps the names q, k, v, q2, k2 to arrays."""
    y = np.asarray(y, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    W = w.shape[0]
    z = causal_conv(y, w)
    B, T, C = z.shape
    dz = np.zeros_like(z)
    c0 = 0
    for name, width, act, norm in _blocks(H, K, V, E):
        zb = z[:, :, c0:c0 + H * width].reshape(B, T, H, width)
        g = np.asarray(grads[name], dtype=np.float64).reshape(B, T, H, width)
        if act == "silu":
            s = _sigmoid(zb)
            a = zb * s
            slope = s + zb * s * _sigmoid(-zb)  # d(z sigmoid z)/dz
        else:
            a = _softplus(zb)
            slope = _sigmoid(zb)
        if norm:
            r = np.sqrt(np.sum(a * a, axis=-1, keepdims=True) + eps)
            # n = a / r:  da = dn / r - a <dn, a> / r^3
            da = g / r - a * np.sum(g * a, axis=-1, keepdims=True) / r ** 3
        else:
            da = g
        dz[:, :, c0:c0 + H * width] = (da * slope).reshape(B, T, H * width)
        c0 += H * width
    dy = np.zeros_like(y)
    dw = np.zeros_like(w)
    for j in range(W):
        shift = W - 1 - j
        if shift < T:
            # z[t] gets w[j] y[t - shift]
            dy[:, :T - shift, :] += w[j] * dz[:, shift:, :]
            dw[j] = np.sum(dz[:, shift:, :] * y[:, :T - shift, :], axis=(0, 1))
    return dy, dw

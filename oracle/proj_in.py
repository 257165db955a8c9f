"""fp64 reference of the mixer's input projection with its epilogue --
TEST INFRASTRUCTURE ONLY (tests, smoke and the bench's CPU baseline use it;
the HIP path never does).

Section "Input projections" and Alg. 2: one GEMM of the normalised block
input u against the stacked projections of q, k, v, q' and k' of every head
gives the channels y that the causal depthwise convolution, the activations
and the normalisations then turn into the operator's inputs (those steps are
`conv_in`'s, reused here unchanged).

Layouts: u [B][T][Dm]; Wp [Ctot][Dm], row c holding the projection of
channel c (y[b, t, c] = sum_d u[b, t, d] Wp[c, d]); channel order as in
`conv_in` (blocks q | k | v | q' | k', each head-major).

The backward is the chain rule: `conv_in`'s backward gives dy, then
du = dy Wp and dWp = sum over tokens of dy^T u.
"""
import numpy as np

from . import conv_in


def project(u, Wp):
    """y[b, t, c] = sum_d u[b, t, d] Wp[c, d] (fp64)."""
    u = np.asarray(u, dtype=np.float64)
    Wp = np.asarray(Wp, dtype=np.float64)
    return np.matmul(u, Wp.T)


def proj_in_fwd(u, Wp, w, H, K, V, E, eps):
    """-> (dict q, k, v, q2, k2 as in conv_in.conv_in_fwd, y [B, T, Ctot])."""
    y = project(u, Wp)
    return conv_in.conv_in_fwd(y, w, H, K, V, E, eps), y


def proj_in_bwd(u, Wp, w, H, K, V, E, eps, grads):
    """Gradients (du [B, T, Dm], dWp [Ctot, Dm], dw [W, Ctot]) of the sum over
    the five outputs of <grads[name], output>."""
    u = np.asarray(u, dtype=np.float64)
    Wp = np.asarray(Wp, dtype=np.float64)
    y = project(u, Wp)
    dy, dw = conv_in.conv_in_bwd(y, w, H, K, V, E, eps, grads)
    du = np.matmul(dy, Wp)
    B, T, C = dy.shape
    dWp = np.matmul(dy.reshape(B * T, C).T, u.reshape(B * T, -1))
    return du, dWp, dw

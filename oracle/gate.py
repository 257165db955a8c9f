"""fp64 reference of the mixer's output side -- TEST INFRASTRUCTURE ONLY.

Alg. 2 (the triadic GDN / sGLA block) ends each head's mixer with
    o_h <- RMSNorm(o_h) (.) sigma(z_h),   z_h = W_g2^h W_g1 u + b_g^h,
where RMSNorm normalises the head's V values by their root mean square and
applies a learned per-channel gain.  The projections that form z are outside
this op: it takes o, the gate pre-activation z and the gain w.  Readings
(the paper gives neither): the gain w has V entries shared by all heads, and
the mean square gets a caller-given eps before the square root.

Plain numpy over rows (the last axis is the head's V values); the backward
is the chain rule written out term by term.
"""
import numpy as np


def _sigmoid(z):
    return 1.0 / (1.0 + np.exp(-z))


def out_gate_fwd(o, z, w, eps):
    """y[..., v] = o[..., v] / sqrt(mean_v o^2 + eps) * w[v] * sigmoid(z[..., v])."""
    o = np.asarray(o, dtype=np.float64)
    z = np.asarray(z, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    inv_rms = 1.0 / np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + eps)
    return o * inv_rms * w * _sigmoid(z)


def out_gate_bwd(o, z, w, eps, dy):
    """Gradients (do, dz, dw) of sum(dy * out_gate_fwd(o, z, w, eps)).

    With r = 1 / sqrt(mean(o^2) + eps), n = o r and s = sigmoid(z):
      y = n w s
      dz = dy w n s (1 - s)
      dw = sum over all rows of dy n s
      dn = dy w s,  and since dn/do = r (I - n n^T / V):
      do = r (dn - n mean(dn n)).
    """
    o = np.asarray(o, dtype=np.float64)
    z = np.asarray(z, dtype=np.float64)
    w = np.asarray(w, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    V = o.shape[-1]
    r = 1.0 / np.sqrt(np.mean(o * o, axis=-1, keepdims=True) + eps)
    n = o * r
    s = _sigmoid(z)
    dz = dy * w * n * s * (1.0 - s)
    dw = np.sum((dy * n * s).reshape(-1, V), axis=0)
    dn = dy * w * s
    do = r * (dn - n * np.sum(dn * n, axis=-1, keepdims=True) / V)
    return do, dz, dw

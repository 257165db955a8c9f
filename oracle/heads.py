"""fp64 reference of the mixer's gate heads -- TEST INFRASTRUCTURE ONLY.

Alg. 2 forms per head h and slice e the forget gate
    alpha_e = exp(-exp(A_e) softplus(x_e + b_e)),   x = W_alpha u,
and the write strength beta = sigmoid(x_beta), x_beta = W_beta u.  The
projections are outside this op; it takes the pre-activations x (per token,
head and slice) and x_beta (per token and head) with the parameters A, b
([H][E]) and returns what the operator consumes: the log-gate
g = log alpha = -exp(A) softplus(x + b) (always <= 0) and beta.  Plain numpy;
the backward is the chain rule written out (softplus' = sigmoid).
"""
import numpy as np


def _softplus(x):
    return np.logaddexp(0.0, x)


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def gate_heads_fwd(x, xb, A, b):
    """x: [..., H, E], xb: [..., H], A, b: [H, E] -> (g [..., H, E], beta [..., H])."""
    x, xb, A, b = (np.asarray(t, dtype=np.float64) for t in (x, xb, A, b))
    g = -np.exp(A) * _softplus(x + b)
    return g, _sigmoid(xb)


def gate_heads_bwd(x, xb, A, b, dg, dbeta):
    """Gradients (dx, dxb, dA, db) of sum(dg * g) + sum(dbeta * beta):
      dx = dg (-exp(A)) sigmoid(x + b),  db = sum over tokens of dx,
      dA = sum over tokens of dg g,      dxb = dbeta beta (1 - beta)."""
    x, xb, A, b, dg, dbeta = (np.asarray(t, dtype=np.float64) for t in (x, xb, A, b, dg, dbeta))
    H, E = A.shape
    g = -np.exp(A) * _softplus(x + b)
    dx = dg * (-np.exp(A)) * _sigmoid(x + b)
    db = np.sum(dx.reshape(-1, H, E), axis=0)
    dA = np.sum((dg * g).reshape(-1, H, E), axis=0)
    # sigmoid' = sigmoid(x) sigmoid(-x) (= beta (1 - beta), without 1 - beta rounding to 0)
    return dx, dbeta * _sigmoid(xb) * _sigmoid(-xb), dA, db

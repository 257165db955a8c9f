"""Independent fp64 formulations of triadic linear attention -- TEST
INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Each function is written from a different statement of the operator in the
paper, so that agreement with the token-by-token C oracle pins it:

* ``flat_joint_key``   -- Eq. gdn3flat: Gated DeltaNet on the joint key
  kappa = k (x) k' of dimension d*E, with the state read as a (d*E) x d matrix,
  a diagonal per-slice decay D_t applied before the erase, and the joint
  query q (x) q'.  For sGLA the erase factor is dropped.
* ``dyadic``           -- ordinary (two-dimensional) gated DeltaNet / gated
  linear attention with a d x d state (Eq. la plus a scalar gate and the delta
  rule); the E = 1, k' = q' = 1 special case of the triadic operator
  (Section 2.2 and Appendix A).
* ``quadratic_sgla``   -- the parallel (attention-like) form of Eq. la3 with
  per-slice forgetting: o_t = sum_{s<=t} (q_t.k_s) [sum_e q'_t[e] k'_s[e]
  prod_{j=s+1..t} a_j[e]] beta_s v_s plus the decayed read of s0.
* ``chunkwise``        -- the chunkwise-parallel form of Appendix A
  (Eq. joint-gram, joint-solve, joint-chunk) in the paper's notation.

Shapes follow the C oracle: q,k [B,T,H,K]; v [B,T,H,V]; q2,k2,g [B,T,H,E];
beta [B,T,H] or None; s0 [B,H,E,K,V] or None.  g is the log-gate (a = exp g).
"""
import numpy as np

SGLA, GDN = 0, 1


def _prep(q, k, v, q2, k2, g, beta, s0):
    q, k, v, q2, k2, g = (np.asarray(x, dtype=np.float64) for x in (q, k, v, q2, k2, g))
    B, T, H, K = q.shape
    V = v.shape[-1]
    E = q2.shape[-1]
    beta = np.ones((B, T, H)) if beta is None else np.asarray(beta, dtype=np.float64)
    s0 = np.zeros((B, H, E, K, V)) if s0 is None else np.asarray(s0, dtype=np.float64)
    return q, k, v, q2, k2, g, beta, s0, (B, T, H, K, V, E)


def flat_joint_key(variant, q, k, v, q2, k2, g, beta=None, s0=None):
    """Eq. gdn3flat with the state as a (E*K) x V matrix; row index e*K + k
    (the joint key k' (x) k in that order matches the [E,K,V] state layout)."""
    q, k, v, q2, k2, g, beta, s0, (B, T, H, K, V, E) = _prep(q, k, v, q2, k2, g, beta, s0)
    o = np.zeros((B, T, H, V))
    sf = np.zeros((B, H, E, K, V))
    eye = np.eye(E * K)
    for b in range(B):
        for h in range(H):
            S = s0[b, h].reshape(E * K, V).copy()
            for t in range(T):
                kap = np.kron(k2[b, t, h], k[b, t, h])          # joint key
                rho = np.kron(q2[b, t, h], q[b, t, h])          # joint query
                D = np.diag(np.repeat(np.exp(g[b, t, h]), K))   # per-slice decay
                bt = beta[b, t, h]
                if variant == GDN:
                    S = (eye - bt * np.outer(kap, kap)) @ D @ S + bt * np.outer(kap, v[b, t, h])
                else:
                    S = D @ S + bt * np.outer(kap, v[b, t, h])
                o[b, t, h] = S.T @ rho
            sf[b, h] = S.reshape(E, K, V)
    return o, sf


def dyadic(variant, q, k, v, g_scalar, beta=None, s0=None):
    """Ordinary gated DeltaNet (variant GDN) or scalar-gated linear attention
    (variant SGLA) with a K x V state per head.  q,k [B,T,H,K]; v [B,T,H,V];
    g_scalar [B,T,H] log-gate; s0 [B,H,K,V]."""
    q, k, v = (np.asarray(x, dtype=np.float64) for x in (q, k, v))
    g_scalar = np.asarray(g_scalar, dtype=np.float64)
    B, T, H, K = q.shape
    V = v.shape[-1]
    beta = np.ones((B, T, H)) if beta is None else np.asarray(beta, dtype=np.float64)
    s0 = np.zeros((B, H, K, V)) if s0 is None else np.asarray(s0, dtype=np.float64)
    o = np.zeros((B, T, H, V))
    sf = np.zeros((B, H, K, V))
    for b in range(B):
        for h in range(H):
            S = s0[b, h].copy()
            for t in range(T):
                kt, bt = k[b, t, h], beta[b, t, h]
                S = np.exp(g_scalar[b, t, h]) * S
                if variant == GDN:
                    S = S - bt * np.outer(kt, kt @ S)
                S = S + bt * np.outer(kt, v[b, t, h])
                o[b, t, h] = S.T @ q[b, t, h]
            sf[b, h] = S
    return o, sf


def quadratic_sgla(q, k, v, q2, k2, g, beta=None, s0=None):
    """Brute-force quadratic form of triadic sGLA (small T only)."""
    q, k, v, q2, k2, g, beta, s0, (B, T, H, K, V, E) = _prep(q, k, v, q2, k2, g, beta, s0)
    a = np.exp(g)
    o = np.zeros((B, T, H, V))
    for b in range(B):
        for h in range(H):
            for t in range(T):
                acc = np.zeros(V)
                # contribution of the initial state, decayed over tokens 1..t
                for e in range(E):
                    dec = np.prod(a[b, : t + 1, h, e])
                    acc += q2[b, t, h, e] * dec * (q[b, t, h] @ s0[b, h, e])
                for s in range(t + 1):
                    mix = 0.0
                    for e in range(E):
                        dec = np.prod(a[b, s + 1: t + 1, h, e])   # empty product = 1
                        mix += q2[b, t, h, e] * k2[b, s, h, e] * dec
                    acc += (q[b, t, h] @ k[b, s, h]) * mix * beta[b, s, h] * v[b, s, h]
                o[b, t, h] = acc
    return o


def chunkwise(variant, q, k, v, q2, k2, g, beta=None, s0=None, chunk=64):
    """Appendix A chunkwise form.  Chunk i covers positions iC+1..iC+C (the
    last chunk may be shorter).  For sGLA (no erase term) the solve reduces
    to T = diag(beta)."""
    q, k, v, q2, k2, g, beta, s0, (B, T, H, K, V, E) = _prep(q, k, v, q2, k2, g, beta, s0)
    o = np.zeros((B, T, H, V))
    sf = np.zeros((B, H, E, K, V))
    for b in range(B):
        for h in range(H):
            S = [s0[b, h, e].copy() for e in range(E)]        # slices S_[i],e
            for c0 in range(0, T, chunk):
                c1 = min(c0 + chunk, T)
                C = c1 - c0
                Q, Kc, Vc = q[b, c0:c1, h], k[b, c0:c1, h], v[b, c0:c1, h]
                Qp, Kp = q2[b, c0:c1, h], k2[b, c0:c1, h]     # Q', K' (C x E)
                bet = beta[b, c0:c1, h]
                Gl = np.cumsum(g[b, c0:c1, h], axis=0)         # log gamma^r_e
                gam = np.exp(Gl)                                # gamma_e (C x E)
                # Gamma_e[r,s] = gamma^r_e / gamma^s_e for r >= s, as exp of a
                # non-positive difference of accumulated log-gates
                low = np.tril(np.ones((C, C)))
                Gam = [np.exp(np.where(low > 0, Gl[:, None, e] - Gl[None, :, e], -np.inf))
                       for e in range(E)]
                R = sum(np.outer(Kp[:, e], Kp[:, e]) * Gam[e] for e in range(E))
                Rq = sum(np.outer(Qp[:, e], Kp[:, e]) * Gam[e] for e in range(E))
                if variant == GDN:
                    Lmat = np.tril(np.diag(bet) @ ((Kc @ Kc.T) * R), -1)
                    Tm = np.linalg.solve(np.eye(C) + Lmat, np.diag(bet))
                else:
                    Tm = np.diag(bet)
                W = sum(np.diag(Kp[:, e] * gam[:, e]) @ Kc @ S[e] for e in range(E))
                U = Tm @ (Vc - W) if variant == GDN else Tm @ Vc
                O = sum(np.diag(Qp[:, e] * gam[:, e]) @ Q @ S[e] for e in range(E))
                O = O + ((Q @ Kc.T) * Rq) @ U
                o[b, c0:c1, h] = O
                gC = gam[-1]
                for e in range(E):
                    tail = np.exp(Gl[-1, e] - Gl[:, e])          # gamma^C / gamma
                    S[e] = gC[e] * S[e] + Kc.T @ np.diag(Kp[:, e] * tail) @ U
            sf[b, h] = np.stack(S)
    return o, sf

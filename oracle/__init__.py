"""fp64 CPU oracle for triadic linear attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never calls it and
shares no code with it.

``fwd``/``bwd``/``step`` wrap the token-by-token C recurrence in
``tla_oracle.c`` (the plain definition of the operator: Eq. forget3, Eq. gdn3,
Eq. la3 and the mixer of Alg. 2).  ``forms`` holds independent numpy
formulations used to pin it (flattened joint key, dyadic special case,
quadratic form, chunkwise form).  ``gate`` is the mixer's output side
(RMSNorm times a sigmoid gate), ``heads`` its gate heads (forget gate and
write strength) and ``conv_in`` its input side after the projection GEMM
(causal depthwise convolution, activations, L2 normalisation), all in numpy.
"""
import ctypes
import os

import numpy as np

from . import build as _build
from .gate import out_gate_bwd, out_gate_fwd  # noqa: F401
from .heads import gate_heads_bwd, gate_heads_fwd  # noqa: F401
from .conv_in import conv_in_bwd, conv_in_fwd  # noqa: F401

SGLA, GDN = 0, 1
_HERE = os.path.dirname(os.path.abspath(__file__))
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    path = os.path.join(_HERE, "liboracle.so")
    src = os.path.join(_HERE, "tla_oracle.c")
    if not os.path.exists(path) or os.path.getmtime(path) < os.path.getmtime(src):
        _build.build()
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I = ctypes.c_int
    lib.oracle_fwd.argtypes = [I] * 7 + [P] * 10
    lib.oracle_fwd.restype = I
    lib.oracle_step.argtypes = [I] * 6 + [P] * 9
    lib.oracle_step.restype = I
    lib.oracle_bwd.argtypes = [I] * 7 + [P] * 18
    lib.oracle_bwd.restype = I
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = I
    _lib = lib
    return lib


def _c(x):
    """C-contiguous float64 copy (or None)."""
    if x is None:
        return None
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _p(x):
    return None if x is None else x.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def fwd(variant, q, k, v, q2, k2, g, beta=None, s0=None):
    """Token-by-token forward.  Shapes: q,k [B,T,H,K]; v [B,T,H,V];
    q2,k2,g [B,T,H,E]; beta [B,T,H] or None; s0 [B,H,E,K,V] or None.
    Returns (o [B,T,H,V], s_final [B,H,E,K,V]) in float64."""
    lib = _load()
    q, k, v, q2, k2, g = map(_c, (q, k, v, q2, k2, g))
    beta, s0 = _c(beta), _c(s0)
    B, T, H, K = q.shape
    V = v.shape[-1]
    E = q2.shape[-1]
    o = np.zeros((B, T, H, V))
    sf = np.zeros((B, H, E, K, V))
    rc = lib.oracle_fwd(variant, B, T, H, K, V, E, _p(q), _p(k), _p(v), _p(q2),
                        _p(k2), _p(g), _p(beta), _p(s0), _p(o), _p(sf))
    if rc != 0:
        raise RuntimeError(f"oracle_fwd failed ({rc})")
    return o, sf


def step(variant, q, k, v, q2, k2, g, beta, state):
    """One token per (n, h).  q,k [N,H,K]; v [N,H,V]; q2,k2,g [N,H,E];
    beta [N,H] or None; state [N,H,E,K,V].  Returns (o, new_state)."""
    lib = _load()
    q, k, v, q2, k2, g = map(_c, (q, k, v, q2, k2, g))
    beta = _c(beta)
    st = np.array(state, dtype=np.float64, order="C", copy=True)
    N, H, K = q.shape
    V = v.shape[-1]
    E = q2.shape[-1]
    o = np.zeros((N, H, V))
    rc = lib.oracle_step(variant, N, H, K, V, E, _p(q), _p(k), _p(v), _p(q2),
                         _p(k2), _p(g), _p(beta), _p(st), _p(o))
    if rc != 0:
        raise RuntimeError(f"oracle_step failed ({rc})")
    return o, st


def bwd(variant, q, k, v, q2, k2, g, beta, s0, dO, dS_final=None):
    """Reverse-mode backward of ``fwd``.  Returns a dict with dq, dk, dv,
    dq2, dk2, dg (log-gate gradient), dbeta (None when beta is None), ds0."""
    lib = _load()
    q, k, v, q2, k2, g, dO = map(_c, (q, k, v, q2, k2, g, dO))
    beta, s0, dS_final = _c(beta), _c(s0), _c(dS_final)
    B, T, H, K = q.shape
    V = v.shape[-1]
    E = q2.shape[-1]
    out = {
        "dq": np.zeros((B, T, H, K)), "dk": np.zeros((B, T, H, K)),
        "dv": np.zeros((B, T, H, V)), "dq2": np.zeros((B, T, H, E)),
        "dk2": np.zeros((B, T, H, E)), "dg": np.zeros((B, T, H, E)),
        "dbeta": np.zeros((B, T, H)) if beta is not None else None,
        "ds0": np.zeros((B, H, E, K, V)),
    }
    rc = lib.oracle_bwd(variant, B, T, H, K, V, E, _p(q), _p(k), _p(v), _p(q2),
                        _p(k2), _p(g), _p(beta), _p(s0), _p(dO), _p(dS_final),
                        _p(out["dq"]), _p(out["dk"]), _p(out["dv"]),
                        _p(out["dq2"]), _p(out["dk2"]), _p(out["dg"]),
                        _p(out["dbeta"]), _p(out["ds0"]))
    if rc != 0:
        raise RuntimeError(f"oracle_bwd failed ({rc})")
    return out

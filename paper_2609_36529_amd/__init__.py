"""Triadic linear attention on MI355X (gfx950): Python binding of ``libtla.so``.

The binding only marshals arguments: every step of the operator runs in the
HIP kernels of the library, behind the C ABI declared in ``include/tla.h``
(``tla_fwd`` / ``tla_bwd`` / ``tla_step``).  PyTorch supplies device memory and
the current HIP stream.  There is no fallback: if the library is missing or a
call fails, an exception is raised.

Shapes (row-major, contiguous):
  q, k [B,T,H,K]; v [B,T,H,V]; q2, k2 [B,T,H,E]; g (log-gates) [B,T,H,E] fp32;
  beta [B,T,H] fp32 or None (sGLA only); states [B,H,E,K,V] fp32.
"""
import ctypes
import os

import torch

SGLA, GDN = 0, 1
F32, BF16 = 0, 1
OP_FWD, OP_BWD = 0, 1

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtla.so")
_lib = None


class Desc(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in
                ("struct_size", "variant", "B", "T", "H", "K", "V", "E", "chunk",
                 "in_dtype", "out_dtype")]


class TLAError(RuntimeError):
    pass


PROF_SLOTS = 16  # kernel kinds of tla_prof_read


def lib():
    """Loads the built HIP library (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2609_36529_amd.build` (hipcc, gfx950)")
    L = ctypes.CDLL(LIB_PATH)
    P, S, I = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    DP = ctypes.POINTER(Desc)
    L.tla_version.restype = I
    L.tla_last_error.restype = ctypes.c_char_p
    L.tla_status_string.restype = ctypes.c_char_p
    L.tla_status_string.argtypes = [I]
    L.tla_supported.argtypes = [DP]
    L.tla_supported.restype = I
    L.tla_workspace_bytes.argtypes = [DP, I]
    L.tla_workspace_bytes.restype = S
    L.tla_saved_bytes.argtypes = [DP]
    L.tla_saved_bytes.restype = S
    L.tla_fwd.argtypes = [DP] + [P] * 12 + [S, P]
    L.tla_fwd.restype = I
    L.tla_bwd.argtypes = [DP] + [P] * 20 + [S, P]
    L.tla_bwd.restype = I
    LL = ctypes.c_longlong
    L.tla_fwd_varlen.argtypes = [DP, P, LL] + [P] * 12 + [S, P]
    L.tla_fwd_varlen.restype = I
    L.tla_bwd_varlen.argtypes = [DP, P, LL] + [P] * 20 + [S, P]
    L.tla_bwd_varlen.restype = I
    L.tla_fwd_noalloc.argtypes = [DP] + [P] * 10 + [P]
    L.tla_fwd_noalloc.restype = I
    L.tla_step.argtypes = [DP] + [P] * 9 + [P]
    L.tla_step.restype = I
    L.tla_out_gate_fwd.argtypes = [I, LL, I, P, P, P, ctypes.c_float, P, P]
    L.tla_out_gate_fwd.restype = I
    L.tla_out_gate_workspace_bytes.argtypes = [LL, I]
    L.tla_out_gate_workspace_bytes.restype = S
    L.tla_out_gate_bwd.argtypes = [I, LL, I, P, P, P, ctypes.c_float, P, P, P, P, P, S, P]
    L.tla_out_gate_bwd.restype = I
    L.tla_gate_heads_fwd.argtypes = [I, LL, I, I, P, P, P, P, P, P, P]
    L.tla_gate_heads_fwd.restype = I
    L.tla_gate_heads_workspace_bytes.argtypes = [LL, I, I]
    L.tla_gate_heads_workspace_bytes.restype = S
    L.tla_gate_heads_bwd.argtypes = [I, LL, I, I] + [P] * 11 + [S, P]
    L.tla_gate_heads_bwd.restype = I
    L.tla_conv_in_fwd.argtypes = [I] * 8 + [ctypes.c_float] + [P] * 8
    L.tla_conv_in_fwd.restype = I
    L.tla_conv_in_workspace_bytes.argtypes = [I] * 7
    L.tla_conv_in_workspace_bytes.restype = S
    L.tla_conv_in_bwd.argtypes = [I] * 8 + [ctypes.c_float] + [P] * 10 + [S, P]
    L.tla_conv_in_bwd.restype = I
    L.tla_proj_in_fwd.argtypes = [I] * 8 + [ctypes.c_float] + [P] * 10
    L.tla_proj_in_fwd.restype = I
    L.tla_proj_in_workspace_bytes.argtypes = [I] * 8
    L.tla_proj_in_workspace_bytes.restype = S
    L.tla_proj_in_bwd.argtypes = [I] * 8 + [ctypes.c_float] + [P] * 13 + [S, P]
    L.tla_proj_in_bwd.restype = I
    L.tla_mfma_rate_flop.argtypes = [I, I, I]
    L.tla_mfma_rate_flop.restype = S
    L.tla_mfma_rate.argtypes = [I, I, I, P, P]
    L.tla_mfma_rate.restype = I
    L.tla_prof_enable.argtypes = [I]
    L.tla_prof_enable.restype = I
    L.tla_prof_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I), I]
    L.tla_prof_read.restype = I
    L.tla_prof_name.argtypes = [I]
    L.tla_prof_name.restype = ctypes.c_char_p
    _lib = L
    return L


def _dtype_code(t):
    if t == torch.float32:
        return F32
    if t == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t}")


def make_desc(variant, B, T, H, K, V, E, chunk, in_dtype, out_dtype):
    d = Desc()
    d.struct_size = ctypes.sizeof(Desc)
    d.variant, d.B, d.T, d.H, d.K, d.V, d.E, d.chunk = variant, B, T, H, K, V, E, chunk
    d.in_dtype, d.out_dtype = in_dtype, out_dtype
    return d


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _check(rc):
    if rc != 0:
        L = lib()
        raise TLAError(f"{L.tla_status_string(rc).decode()} ({L.tla_last_error().decode()})")


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _need(t, name, dtype=None, device=None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    return t


def _shape(t, name, shape):
    """Raises unless tensor t (if given) has exactly `shape`."""
    if t is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return t


def _buffer(t, name, nbytes, device):
    """A caller-supplied byte buffer: a contiguous device tensor of at least
    nbytes bytes (any element type)."""
    if t is None:
        return None
    _need(t, name, None, device)
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes, the call needs {nbytes}")
    return t


def _check_inputs(q, k, v, q2, k2, g, beta, s0, packed_B=None):
    """Every operator input: device, contiguity, element type and shape
    against q [B, T, H, K], v [.., V], q2 [.., E].  Raises before any launch.
    packed_B: the number of packed sequences (states are [packed_B, H, E, K, V])."""
    if q.dim() != 4 or v.dim() != 4 or q2.dim() != 4:
        raise ValueError("q, v and q2 must be 4-d: [B, T, H, K], [B, T, H, V], [B, T, H, E]")
    dev, dt = q.device, q.dtype
    _dtype_code(dt)
    B, T, H, K = q.shape
    V, E = v.shape[-1], q2.shape[-1]
    for name, t, last in (("q", q, K), ("k", k, K), ("v", v, V), ("q2", q2, E), ("k2", k2, E)):
        _need(t, name, dt, dev)
        _shape(t, name, (B, T, H, last))
    _shape(_need(g, "g", torch.float32, dev), "g", (B, T, H, E))
    _shape(_need(beta, "beta", torch.float32, dev), "beta", (B, T, H))
    nb = B if packed_B is None else packed_B
    _shape(_need(s0, "s0", torch.float32, dev), "s0", (nb, H, E, K, V))
    return dev, dt


def describe(variant, q, v, q2, chunk, out_dtype=None, cu_seqlens=None, max_seqlen=None):
    """Descriptor of a call; with cu_seqlens (packed sequences, q is
    [1, total, H, K]) B is the number of sequences and T = max_seqlen."""
    B, T, H, K = q.shape
    if cu_seqlens is not None:
        if B != 1 or max_seqlen is None:
            raise ValueError("packed sequences need q of shape [1, total, H, K] and max_seqlen")
        B, T = cu_seqlens.numel() - 1, int(max_seqlen)
    return make_desc(variant, B, T, H, K, v.shape[-1], q2.shape[-1], chunk, _dtype_code(q.dtype),
                     _dtype_code(out_dtype if out_dtype is not None else q.dtype))


def _cu(cu_seqlens, dev):
    if cu_seqlens is None:
        return None
    _need(cu_seqlens, "cu_seqlens", torch.int32, dev)
    return cu_seqlens


def supported(desc):
    return bool(lib().tla_supported(ctypes.byref(desc)))


def workspace_bytes(desc, op):
    return int(lib().tla_workspace_bytes(ctypes.byref(desc), op))


def saved_bytes(desc):
    return int(lib().tla_saved_bytes(ctypes.byref(desc)))


def fwd(variant, q, k, v, q2, k2, g, beta=None, s0=None, chunk=64, out_dtype=None,
        want_final=True, training=False, o=None, s_final=None, ws=None, saved=None,
        cu_seqlens=None, max_seqlen=None):
    """Chunkwise forward.  Returns (o, s_final or None, saved or None).
    With cu_seqlens (int32 device tensor of N + 1 offsets) the inputs hold N
    packed sequences, [1, total, H, .], each with its own state (s0 and
    s_final [N, H, E, K, V]); max_seqlen is the longest length."""
    cu = _cu(cu_seqlens, q.device)
    dev, dt = _check_inputs(q, k, v, q2, k2, g, beta, s0,
                            None if cu is None else cu.numel() - 1)
    desc = describe(variant, q, v, q2, chunk, out_dtype, cu, max_seqlen)
    B, T = desc.B, desc.T
    H, K = q.shape[2], q.shape[3]
    V, E = v.shape[-1], q2.shape[-1]
    odt = out_dtype or dt
    if o is None:
        o = torch.empty(q.shape[:3] + (V,), dtype=odt, device=dev)
    _shape(_need(o, "o", odt, dev), "o", q.shape[:3] + (V,))
    if want_final and s_final is None:
        s_final = torch.empty((B, H, E, K, V), dtype=torch.float32, device=dev)
    if want_final:
        _shape(_need(s_final, "s_final", torch.float32, dev), "s_final", (B, H, E, K, V))
    if training:
        if saved is None:
            saved = torch.empty(max(saved_bytes(desc), 1), dtype=torch.uint8, device=dev)
        _buffer(saved, "saved", saved_bytes(desc), dev)
    elif ws is None:
        ws = torch.empty(max(workspace_bytes(desc, OP_FWD), 1), dtype=torch.uint8, device=dev)
    _buffer(ws, "ws", 0 if training else workspace_bytes(desc, OP_FWD), dev)
    args = (_ptr(q), _ptr(k), _ptr(v), _ptr(q2), _ptr(k2), _ptr(g), _ptr(beta), _ptr(s0), _ptr(o),
            _ptr(s_final if want_final else None), _ptr(saved if training else None), _ptr(ws),
            0 if ws is None else ws.numel() * ws.element_size(), _stream(dev))
    if cu is None:
        rc = lib().tla_fwd(ctypes.byref(desc), *args)
    else:
        rc = lib().tla_fwd_varlen(ctypes.byref(desc), _ptr(cu), q.shape[1], *args)
    _check(rc)
    return o, (s_final if want_final else None), (saved if training else None)


def bwd(variant, q, k, v, q2, k2, g, beta, s0, dO, saved, dS_final=None, chunk=64,
        out_dtype=None, want_ds0=True, ws=None, grads=None, cu_seqlens=None, max_seqlen=None):
    """Backward of a training forward.  Returns a dict of gradients
    (dq, dk, dv, dq2, dk2 in out_dtype (default: the input dtype); dg, dbeta or
    None, ds0 or None in fp32).  cu_seqlens / max_seqlen as for fwd."""
    cu = _cu(cu_seqlens, q.device)
    dev, dt = _check_inputs(q, k, v, q2, k2, g, beta, s0,
                            None if cu is None else cu.numel() - 1)
    gt = out_dtype or dt
    desc = describe(variant, q, v, q2, chunk, gt, cu, max_seqlen)
    B = desc.B
    H, K = q.shape[2], q.shape[3]
    V, E = v.shape[-1], q2.shape[-1]
    _shape(_need(dO, "dO", dt, dev), "dO", v.shape)
    _shape(_need(dS_final, "dS_final", torch.float32, dev), "dS_final", (B, H, E, K, V))
    if saved is None:
        raise ValueError("bwd needs the `saved` buffer of a training forward")
    _buffer(saved, "saved", saved_bytes(desc), dev)
    if grads is None:
        grads = {
            "dq": torch.empty_like(q, dtype=gt), "dk": torch.empty_like(k, dtype=gt),
            "dv": torch.empty_like(v, dtype=gt), "dq2": torch.empty_like(q2, dtype=gt),
            "dk2": torch.empty_like(k2, dtype=gt),
            "dg": torch.empty(q.shape[:3] + (E,), dtype=torch.float32, device=dev),
            "dbeta": None if beta is None else torch.empty(q.shape[:3], dtype=torch.float32, device=dev),
            "ds0": torch.empty((B, H, E, K, V), dtype=torch.float32, device=dev) if want_ds0 else None,
        }
    expect = {"dq": (q.shape, gt), "dk": (q.shape, gt), "dv": (v.shape, gt), "dq2": (q2.shape, gt),
              "dk2": (q2.shape, gt), "dg": (q2.shape, torch.float32),
              "dbeta": (q.shape[:3], torch.float32), "ds0": ((B, H, E, K, V), torch.float32)}
    for key, (shp, gdt) in expect.items():
        _shape(_need(grads.get(key), key, gdt, dev), key, shp)
    if (beta is None) != (grads.get("dbeta") is None):
        raise ValueError("grads['dbeta'] must be given exactly when beta is")
    if ws is None:
        ws = torch.empty(max(workspace_bytes(desc, OP_BWD), 1), dtype=torch.uint8, device=dev)
    _buffer(ws, "ws", workspace_bytes(desc, OP_BWD), dev)
    args = (_ptr(q), _ptr(k), _ptr(v), _ptr(q2), _ptr(k2), _ptr(g), _ptr(beta), _ptr(s0), _ptr(dO),
            _ptr(dS_final), _ptr(saved), *[_ptr(grads.get(key)) for key in expect], _ptr(ws),
            ws.numel() * ws.element_size(), _stream(dev))
    if cu is None:
        rc = lib().tla_bwd(ctypes.byref(desc), *args)
    else:
        rc = lib().tla_bwd_varlen(ctypes.byref(desc), _ptr(cu), q.shape[1], *args)
    _check(rc)
    return grads


NOALLOC_SCRATCH_BYTES = 64 << 20  # TLA_NOALLOC_SCRATCH_BYTES


def fwd_noalloc(variant, q, k, v, q2, k2, g, beta=None, s0=None, chunk=64, out_dtype=None,
                o=None, s_final=None):
    """Inference forward through tla_fwd_noalloc: the library's static device
    scratch replaces the caller workspace.  o and s_final may be given (then
    nothing at all is allocated); returns (o, s_final or None)."""
    dev, dt = _check_inputs(q, k, v, q2, k2, g, beta, s0)
    desc = describe(variant, q, v, q2, chunk, out_dtype)
    B, T, H, K = q.shape
    V, E = v.shape[-1], q2.shape[-1]
    odt = out_dtype or dt
    if o is None:
        o = torch.empty(q.shape[:3] + (V,), dtype=odt, device=dev)
    _shape(_need(o, "o", odt, dev), "o", q.shape[:3] + (V,))
    _shape(_need(s_final, "s_final", torch.float32, dev), "s_final", (B, H, E, K, V))
    _check(lib().tla_fwd_noalloc(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(q2), _ptr(k2),
                                 _ptr(g), _ptr(beta), _ptr(s0), _ptr(o), _ptr(s_final),
                                 _stream(dev)))
    return o, s_final


class TriadicAttention(torch.autograd.Function):
    """Autograd wrapper of one training forward (tla_fwd with a `saved`
    buffer) and its backward (tla_bwd).  Inputs as for fwd(); returns
    (o, s_final).  Gradients flow to q, k, v, q2, k2, g, beta and s0 (those
    given); those of q, k, v, q2, k2 have out_dtype (default: the operand
    type), as o does.  The `saved` buffer of the forward is held until the
    backward."""

    @staticmethod
    def forward(ctx, q, k, v, q2, k2, g, beta, s0, variant, chunk, out_dtype):
        o, s_final, saved = fwd(variant, q, k, v, q2, k2, g, beta, s0, chunk=chunk,
                                out_dtype=out_dtype, training=True)
        ctx.save_for_backward(q, k, v, q2, k2, g, beta, s0)
        ctx.saved_buffer = saved
        ctx.variant, ctx.chunk, ctx.out_dtype = variant, chunk, out_dtype
        return o, s_final

    @staticmethod
    def backward(ctx, do, dsf):
        q, k, v, q2, k2, g, beta, s0 = ctx.saved_tensors
        if do is None:
            do = torch.zeros(v.shape, dtype=q.dtype, device=q.device)
        do = do.to(q.dtype).contiguous()
        dsf = None if dsf is None else dsf.float().contiguous()
        gr = bwd(ctx.variant, q, k, v, q2, k2, g, beta, s0, do, ctx.saved_buffer, dS_final=dsf,
                 chunk=ctx.chunk, out_dtype=ctx.out_dtype or q.dtype, want_ds0=s0 is not None)
        ctx.saved_buffer = None
        return (gr["dq"], gr["dk"], gr["dv"], gr["dq2"], gr["dk2"], gr["dg"], gr["dbeta"],
                gr["ds0"], None, None, None)


def attention(variant, q, k, v, q2, k2, g, beta=None, s0=None, chunk=64, out_dtype=None):
    """Differentiable triadic linear attention: (o, s_final) with autograd
    support through TriadicAttention (training forward + tla_bwd)."""
    return TriadicAttention.apply(q, k, v, q2, k2, g, beta, s0, variant, chunk, out_dtype)


def step(variant, q, k, v, q2, k2, g, beta, state, out_dtype=None, o=None):
    """One decode token per (sequence, head); updates `state` in place.
    q, k [N,H,K]; v [N,H,V]; q2, k2, g [N,H,E]; beta [N,H] or None."""
    dev = q.device
    if q.dim() != 3 or v.dim() != 3 or q2.dim() != 3:
        raise ValueError("q, v and q2 must be 3-d: [N, H, K], [N, H, V], [N, H, E]")
    N, H, K = q.shape
    V, E = v.shape[-1], q2.shape[-1]
    for name, t, last in (("q", q, K), ("k", k, K), ("v", v, V), ("q2", q2, E), ("k2", k2, E)):
        _shape(_need(t, name, q.dtype, dev), name, (N, H, last))
    _shape(_need(g, "g", torch.float32, dev), "g", (N, H, E))
    _shape(_need(beta, "beta", torch.float32, dev), "beta", (N, H))
    if state is None:
        raise ValueError("step needs the state tensor")
    _shape(_need(state, "state", torch.float32, dev), "state", (N, H, E, K, V))
    desc = make_desc(variant, N, 1, H, K, V, E, 16, _dtype_code(q.dtype),
                     _dtype_code(out_dtype or q.dtype))
    if o is None:
        o = torch.empty((N, H, V), dtype=out_dtype or q.dtype, device=dev)
    _shape(_need(o, "o", out_dtype or q.dtype, dev), "o", (N, H, V))
    rc = lib().tla_step(ctypes.byref(desc), _ptr(q), _ptr(k), _ptr(v), _ptr(q2), _ptr(k2), _ptr(g),
                        _ptr(beta), _ptr(state), _ptr(o), _stream(dev))
    _check(rc)
    return o


def out_gate_fwd(o, z, w, eps=1e-6, y=None):
    """The mixer's output side (Alg. 2): y = o / sqrt(mean(o^2) + eps) * w * sigmoid(z)
    over the last axis (V values of one head), for o, z of any leading shape
    (bf16 or fp32, contiguous), gain w fp32 [V].  Runs tla_out_gate_fwd."""
    _need(o, "o")
    V = o.shape[-1]
    dev = o.device
    dt = _dtype_code(o.dtype)
    _need(z, "z", o.dtype, dev)
    _need(w, "w", torch.float32, dev)
    if tuple(z.shape) != tuple(o.shape) or tuple(w.shape) != (V,):
        raise ValueError("z must match o, w must be [V]")
    if y is None:
        y = torch.empty_like(o)
    rows = o.numel() // V if V else 0
    _check(lib().tla_out_gate_fwd(dt, rows, V, _ptr(o), _ptr(z), _ptr(w), float(eps), _ptr(y),
                                  _stream(dev)))
    return y


def out_gate_bwd(o, z, w, dy, eps=1e-6):
    """Gradients (d_o, dz, dw) of the output gate for upstream dy (tla_out_gate_bwd;
    dw summed over all rows in a fixed order)."""
    _need(o, "o")
    V = o.shape[-1]
    dev = o.device
    dt = _dtype_code(o.dtype)
    for t, nm in ((z, "z"), (dy, "dy")):
        _need(t, nm, o.dtype, dev)
    _need(w, "w", torch.float32, dev)
    rows = o.numel() // V if V else 0
    d_o, dz = torch.empty_like(o), torch.empty_like(o)
    dw = torch.empty(V, dtype=torch.float32, device=dev)
    L = lib()
    ws = torch.empty(max(L.tla_out_gate_workspace_bytes(rows, V), 256), dtype=torch.uint8, device=dev)
    _check(L.tla_out_gate_bwd(dt, rows, V, _ptr(o), _ptr(z), _ptr(w), float(eps), _ptr(dy), _ptr(d_o),
                              _ptr(dz), _ptr(dw), _ptr(ws), ws.numel(), _stream(dev)))
    return d_o, dz, dw


def gate_heads_fwd(x, xb, A, b):
    """The mixer's gate heads (Alg. 2): g = -exp(A) softplus(x + b) (the log
    forget gate, fp32) and beta = sigmoid(xb) (fp32, None if xb is None), for
    x [..., H, E], xb [..., H] (bf16 or fp32, contiguous), A, b fp32 [H, E].
    Runs tla_gate_heads_fwd."""
    _need(x, "x")
    dev = x.device
    dt = _dtype_code(x.dtype)
    H, E = A.shape
    _need(A, "A", torch.float32, dev)
    _need(b, "b", torch.float32, dev)
    _need(xb, "xb", x.dtype, dev)
    if tuple(x.shape[-2:]) != (H, E) or tuple(b.shape) != (H, E):
        raise ValueError("x must end in [H, E] and b must be [H, E] like A")
    if xb is not None and tuple(xb.shape) != tuple(x.shape[:-1]):
        raise ValueError("xb must be x's shape without the last axis")
    tokens = x.numel() // (H * E)
    g = torch.empty(x.shape, dtype=torch.float32, device=dev)
    beta = None if xb is None else torch.empty(xb.shape, dtype=torch.float32, device=dev)
    _check(lib().tla_gate_heads_fwd(dt, tokens, H, E, _ptr(x), _ptr(xb), _ptr(A), _ptr(b), _ptr(g),
                                    _ptr(beta), _stream(dev)))
    return g, beta


def gate_heads_bwd(x, xb, A, b, dg, dbeta):
    """Gradients (dx, dxb, dA, db) of the gate heads for upstream dg, dbeta
    (fp32; dbeta and dxb None when xb is None); dA, db are summed over all
    tokens in a fixed order.  Runs tla_gate_heads_bwd."""
    _need(x, "x")
    dev = x.device
    dt = _dtype_code(x.dtype)
    H, E = A.shape
    _need(A, "A", torch.float32, dev)
    _need(b, "b", torch.float32, dev)
    _need(xb, "xb", x.dtype, dev)
    _need(dg, "dg", torch.float32, dev)
    _need(dbeta, "dbeta", torch.float32, dev)
    if tuple(dg.shape) != tuple(x.shape) or (xb is not None and dbeta is not None
                                            and tuple(dbeta.shape) != tuple(xb.shape)):
        raise ValueError("dg must match x and dbeta must match xb")
    tokens = x.numel() // (H * E)
    dx = torch.empty_like(x)
    dxb = None if xb is None else torch.empty_like(xb)
    dA = torch.empty((H, E), dtype=torch.float32, device=dev)
    db = torch.empty((H, E), dtype=torch.float32, device=dev)
    L = lib()
    ws = torch.empty(max(L.tla_gate_heads_workspace_bytes(tokens, H, E), 256), dtype=torch.uint8,
                     device=dev)
    _check(L.tla_gate_heads_bwd(dt, tokens, H, E, _ptr(x), _ptr(xb), _ptr(A), _ptr(b), _ptr(dg),
                                _ptr(dbeta), _ptr(dx), _ptr(dxb), _ptr(dA), _ptr(db), _ptr(ws),
                                ws.numel(), _stream(dev)))
    return dx, dxb, dA, db


def _conv_shape(y, w, H, K, V, E):
    _need(y, "y")
    dev = y.device
    if y.dim() != 3 or y.shape[-1] != H * (2 * K + V + 2 * E):
        raise ValueError("y must be [B, T, H (2K + V + 2E)]")
    _need(w, "w", torch.float32, dev)
    if w.dim() != 2 or w.shape[1] != y.shape[-1]:
        raise ValueError("w must be [W, Ctot]")
    return y.shape[0], y.shape[1], w.shape[0], dev


def conv_in_fwd(y, w, H, K, V, E, eps=1e-6):
    """The mixer's input side after the projection GEMM (section "Input
    projections", Alg. 2): causal depthwise convolution with taps w [W, Ctot]
    over y [B, T, Ctot] (channel blocks q | k | v | q' | k', head-major), SiLU
    on q, k, v, softplus on q', k', L2 normalisation of q, k, q', k'.
    Returns (q, k, v, q2, k2) as [B, T, H, .] tensors of y's dtype.  Runs
    tla_conv_in_fwd."""
    B, T, W, dev = _conv_shape(y, w, H, K, V, E)
    outs = [torch.empty((B, T, H, d), dtype=y.dtype, device=dev) for d in (K, K, V, E, E)]
    _check(lib().tla_conv_in_fwd(_dtype_code(y.dtype), B, T, H, K, V, E, W, float(eps), _ptr(y), _ptr(w),
                                 *[_ptr(o) for o in outs], _stream(dev)))
    return tuple(outs)


def conv_in_bwd(y, w, H, K, V, E, grads, eps=1e-6):
    """Gradients (dy, dw) of the input side for the outputs' gradients
    grads = (dq, dk, dv, dq2, dk2); dw is summed over all tokens in a fixed
    order.  Runs tla_conv_in_bwd."""
    B, T, W, dev = _conv_shape(y, w, H, K, V, E)
    for gr, d, nm in zip(grads, (K, K, V, E, E), ("dq", "dk", "dv", "dq2", "dk2")):
        _need(gr, nm, y.dtype, dev)
        if tuple(gr.shape) != (B, T, H, d):
            raise ValueError(f"{nm} must be [B, T, H, {d}]")
    dy = torch.empty_like(y)
    dw = torch.empty_like(w)
    L = lib()
    ws = torch.empty(max(L.tla_conv_in_workspace_bytes(B, T, H, K, V, E, W), 256), dtype=torch.uint8,
                     device=dev)
    _check(L.tla_conv_in_bwd(_dtype_code(y.dtype), B, T, H, K, V, E, W, float(eps), _ptr(y), _ptr(w),
                             *[_ptr(g) for g in grads], _ptr(dy), _ptr(dw), _ptr(ws), ws.numel(),
                             _stream(dev)))
    return dy, dw


def _proj_shape(u, Wp, w, H, K, V, E):
    _need(u, "u", torch.bfloat16)
    dev = u.device
    _need(Wp, "Wp", torch.bfloat16, dev)
    _need(w, "w", torch.float32, dev)
    C = H * (2 * K + V + 2 * E)
    if u.dim() != 3 or Wp.dim() != 2 or tuple(Wp.shape) != (C, u.shape[-1]):
        raise ValueError("u must be [B, T, Dm] and Wp [H (2K + V + 2E), Dm]")
    if w.dim() != 2 or w.shape[1] != C:
        raise ValueError("w must be [W, Ctot]")
    return u.shape[0], u.shape[1], u.shape[2], w.shape[0], C, dev


def proj_in_fwd(u, Wp, w, H, K, V, E, eps=1e-6, keep_y=False):
    """The mixer's input projection with the input side fused (section
    "Input projections", Alg. 2): y = u Wp^T for every channel of q, k, v,
    q', k', then the causal convolution with taps w [W, Ctot], SiLU /
    softplus and the L2 normalisations, in one kernel (bf16 operands).
    Returns (q, k, v, q2, k2, y); y [B, T, Ctot] (bf16) only with keep_y,
    else None.  Runs tla_proj_in_fwd."""
    B, T, Dm, W, C, dev = _proj_shape(u, Wp, w, H, K, V, E)
    outs = [torch.empty((B, T, H, d), dtype=torch.bfloat16, device=dev) for d in (K, K, V, E, E)]
    y = torch.empty((B, T, C), dtype=torch.bfloat16, device=dev) if keep_y else None
    _check(lib().tla_proj_in_fwd(B, T, Dm, H, K, V, E, W, float(eps), _ptr(u), _ptr(Wp), _ptr(w),
                                 *[_ptr(o) for o in outs], _ptr(y), _stream(dev)))
    return (*outs, y)


def proj_in_bwd(u, Wp, w, y, H, K, V, E, grads, eps=1e-6):
    """Gradients (du, dWp, dw) of the fused input projection for the
    outputs' gradients grads = (dq, dk, dv, dq2, dk2), given the forward's y
    (proj_in_fwd with keep_y); du is bf16, dWp and dw fp32, every sum over
    tokens in a fixed order.  Runs tla_proj_in_bwd."""
    B, T, Dm, W, C, dev = _proj_shape(u, Wp, w, H, K, V, E)
    _need(y, "y", torch.bfloat16, dev)
    if tuple(y.shape) != (B, T, C):
        raise ValueError("y must be [B, T, Ctot]")
    for gr, d, nm in zip(grads, (K, K, V, E, E), ("dq", "dk", "dv", "dq2", "dk2")):
        _need(gr, nm, torch.bfloat16, dev)
        if tuple(gr.shape) != (B, T, H, d):
            raise ValueError(f"{nm} must be [B, T, H, {d}]")
    du = torch.empty_like(u)
    dWp = torch.empty(Wp.shape, dtype=torch.float32, device=dev)
    dw = torch.empty_like(w)
    L = lib()
    ws = torch.empty(max(L.tla_proj_in_workspace_bytes(B, T, Dm, H, K, V, E, W), 256),
                     dtype=torch.uint8, device=dev)
    _check(L.tla_proj_in_bwd(B, T, Dm, H, K, V, E, W, float(eps), _ptr(u), _ptr(Wp), _ptr(w), _ptr(y),
                             *[_ptr(g) for g in grads], _ptr(du), _ptr(dWp), _ptr(dw), _ptr(ws),
                             ws.numel(), _stream(dev)))
    return du, dWp, dw


def mfma_rate(shape, blocks, iters, sink):
    """Launch the MFMA-rate diagnostic (shape 0: 16x16x32, 1: 32x32x16 bf16)
    on the current stream; returns its FLOP count.  sink: a float32 device
    tensor of at least blocks * 256 elements.  Runs tla_mfma_rate."""
    _need(sink, "sink", torch.float32)
    if sink.numel() < blocks * 256:
        raise ValueError("sink needs blocks * 256 floats")
    L = lib()
    _check(L.tla_mfma_rate(shape, blocks, iters, _ptr(sink), _stream(sink.device)))
    return L.tla_mfma_rate_flop(shape, blocks, iters)


def prof_enable(on=True):
    """Start (clearing old records) or stop per-kernel HIP-event timing."""
    _check(lib().tla_prof_enable(1 if on else 0))


def prof_read():
    """{kernel name: (total ms, launches)} for the launches since prof_enable()."""
    L = lib()
    tot = (ctypes.c_double * PROF_SLOTS)()
    cnt = (ctypes.c_int * PROF_SLOTS)()
    _check(L.tla_prof_read(tot, cnt, PROF_SLOTS))
    return {L.tla_prof_name(i).decode(): (tot[i], cnt[i]) for i in range(PROF_SLOTS)}

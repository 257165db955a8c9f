"""CPU tests of the C ABI: the library loads without a GPU, exports every
function that include/tla.h declares, and rejects bad arguments on the host
(with status codes) before anything reaches the device.  Pointers passed here
are fake addresses; every call is built to fail validation."""
import ctypes
import os
import re

import pytest

import paper_2609_36529_amd as tla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tla.h")

OK, E_NULL, E_SHAPE, E_UNSUP, E_ALIGN, E_WS, E_ALIAS, E_DEVICE = range(8)
FAKE = 0x7f0000000000  # 16-byte aligned fake device address; never dereferenced


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^[A-Za-z_][\w\s\*]*?\b(tla_\w+)\(", text, flags=re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("tla_fwd", "tla_bwd", "tla_step", "tla_workspace_bytes", "tla_saved_bytes",
              "tla_status_string", "tla_last_error", "tla_version", "tla_supported"):
        assert n in names


def test_library_exports_every_declared_symbol():
    L = tla.lib()
    for n in declared_functions():
        assert hasattr(L, n), n


def test_version_and_status_strings():
    L = tla.lib()
    assert L.tla_version() == 1
    for code in range(8):
        assert L.tla_status_string(code)
    assert b"unknown" in L.tla_status_string(99)


def desc(**kw):
    base = dict(variant=tla.GDN, B=2, T=100, H=2, K=128, V=128, E=8, chunk=64,
                in_dtype=tla.BF16, out_dtype=tla.F32)
    base.update(kw)
    return tla.make_desc(base["variant"], base["B"], base["T"], base["H"], base["K"], base["V"],
                         base["E"], base["chunk"], base["in_dtype"], base["out_dtype"])


def fwd_call(d, q=FAKE, k=FAKE + 0x100000, v=FAKE + 0x200000, q2=FAKE + 0x300000,
             k2=FAKE + 0x400000, g=FAKE + 0x500000, beta=FAKE + 0x600000, s0=None,
             o=FAKE + 0x1000000, sf=None, saved=None, ws=FAKE + 0x2000000, ws_bytes=None):
    L = tla.lib()
    if ws_bytes is None:
        ws_bytes = 1 << 40
    P = ctypes.c_void_p
    return L.tla_fwd(ctypes.byref(d), P(q), P(k), P(v), P(q2), P(k2), P(g), P(beta), P(s0), P(o),
                     P(sf), P(saved), P(ws), ws_bytes, None)


def last_error():
    return tla.lib().tla_last_error().decode()


def test_null_desc():
    L = tla.lib()
    P = ctypes.c_void_p
    assert L.tla_fwd(None, *([P(FAKE)] * 11), P(FAKE), 1 << 30, None) == E_NULL
    assert L.tla_workspace_bytes(None, 0) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(variant=7), E_SHAPE),
    (dict(in_dtype=5), E_SHAPE),
    (dict(B=0), E_SHAPE),
    (dict(T=-1), E_SHAPE),
    (dict(K=48), E_UNSUP),
    (dict(V=100), E_UNSUP),
    (dict(V=2048), E_UNSUP),
    (dict(E=3), E_UNSUP),
    (dict(chunk=128), E_UNSUP),
    (dict(K=64, chunk=64, E=2), E_UNSUP),
    (dict(in_dtype=tla.F32, E=16), E_UNSUP),   # fp32 plan exceeds the LDS budget
])
def test_bad_shapes(kw, code):
    assert fwd_call(desc(**kw)) == code
    assert last_error()


def test_struct_size_checked():
    d = desc()
    d.struct_size = 12
    assert fwd_call(d) == E_SHAPE


def test_required_pointers():
    assert fwd_call(desc(), q=None) == E_NULL
    assert fwd_call(desc(), o=None) == E_NULL
    assert fwd_call(desc(variant=tla.GDN), beta=None) == E_NULL


def test_alignment():
    assert fwd_call(desc(), k=FAKE + 0x100008) == E_ALIGN
    assert fwd_call(desc(), ws=FAKE + 0x2000004) == E_ALIGN


def test_workspace_size():
    d = desc()
    need = tla.workspace_bytes(d, tla.OP_FWD)
    assert need > 0
    assert fwd_call(d, ws_bytes=need - 1) == E_WS
    assert fwd_call(d, ws=None) == E_WS


def test_aliasing():
    assert fwd_call(desc(), o=FAKE) == E_ALIAS                  # o overlaps q
    assert fwd_call(desc(), sf=FAKE + 0x400000) == E_ALIAS      # s_final overlaps k2
    assert fwd_call(desc(), ws=FAKE + 0x1000000) == E_ALIAS     # workspace overlaps o


def test_bwd_validation():
    L = tla.lib()
    P = ctypes.c_void_p
    d = desc()
    base = [P(FAKE + i * 0x1000000) for i in range(19)]

    def call(args, ws_bytes=1 << 40):
        return L.tla_bwd(ctypes.byref(d), *args, P(FAKE + 0x40000000), ws_bytes, None)
    # dbeta (index 17) must be given exactly when beta (index 6) is
    args = list(base)
    args[17] = None
    assert call(args) == E_NULL
    args = list(base)
    args[9] = P(FAKE + 8)  # dS_final misaligned
    assert call(args) == E_ALIGN
    assert call(base, ws_bytes=16) == E_WS
    args = list(base)
    args[12] = args[0]  # dk aliases q
    assert call(args) == E_ALIAS


def test_step_validation():
    L = tla.lib()
    P = ctypes.c_void_p
    d = desc(B=4)
    ptrs = [P(FAKE + i * 0x100000) for i in range(9)]
    assert L.tla_step(ctypes.byref(d), *ptrs[:6], None, *ptrs[7:], None) == E_NULL  # GDN without beta
    ptrs2 = list(ptrs)
    ptrs2[8] = ptrs2[7]  # o aliases the state
    assert L.tla_step(ctypes.byref(d), *ptrs2, None) == E_ALIAS
    assert L.tla_step(ctypes.byref(desc(K=128, E=2)), *ptrs, None) == E_UNSUP


def test_size_queries():
    d = desc(B=4, T=4096, H=8)
    ws_f, ws_b, sv = (tla.workspace_bytes(d, tla.OP_FWD), tla.workspace_bytes(d, tla.OP_BWD),
                      tla.saved_bytes(d))
    nch = 4 * 8 * 64
    # forward workspace: per-chunk coefficient vectors, gamma^C and the bf16
    # operand tiles (M, Tu as hi + lo pairs, row-major; K^T, Q^T)
    assert ws_f == nch * (3 * 8 * 64 * 4 + 8 * 4 + (4 * 64 * 64 + 2 * 128 * 64) * 2)
    # saved: bf16 chunk-start states, fp32 U and V - W, the same prep terms
    # and, for GDN, the fp32 (I + L)^{-1} of every chunk for the backward
    assert sv == nch * (8 * 128 * 128 * 2 + 2 * 64 * 128 * 4 + 64 * 64 * 4) + ws_f
    assert ws_b > ws_f > 0
    assert tla.supported(d)
    assert not tla.supported(desc(K=48))


def test_varlen_validation():
    """Packed-sequence entry points: offsets are required, 4-byte aligned, and
    the packed length may not exceed B * T (T is the longest sequence)."""
    L = tla.lib()
    P = ctypes.c_void_p
    d = desc(B=3, T=100)
    ptrs = [P(FAKE + i * 0x1000000) for i in range(12)]

    def fcall(cu, total):
        return L.tla_fwd_varlen(ctypes.byref(d), cu, total, *ptrs, 1 << 40, None)

    def bcall(cu, total):
        return L.tla_bwd_varlen(ctypes.byref(d), cu, total, *[P(FAKE + i * 0x1000000)
                                                             for i in range(20)], 1 << 40, None)
    assert fcall(None, 10) == E_NULL
    assert bcall(None, 10) == E_NULL
    assert fcall(P(FAKE + 0x70000002), 10) == E_ALIGN
    assert fcall(P(FAKE + 0x70000000), 301) == E_SHAPE
    assert fcall(P(FAKE + 0x70000000), -1) == E_SHAPE
    assert bcall(P(FAKE + 0x70000000), 301) == E_SHAPE


def test_out_gate_validation():
    """Output gate: dtype, V, eps, required pointers, alignment, aliasing and
    workspace are checked on the host (fake addresses, nothing launched)."""
    L = tla.lib()
    P = ctypes.c_void_p
    o, z, w, y = (P(FAKE + i * 0x1000000) for i in range(4))
    rows, V = 1000, 128

    def fwd(dtype=tla.BF16, rows_=rows, V_=V, eps=1e-6, **kw):
        a = dict(o=o, z=z, w=w, y=y)
        a.update(kw)
        return L.tla_out_gate_fwd(dtype, rows_, V_, a["o"], a["z"], a["w"], eps, a["y"], None)
    assert fwd(dtype=7) == E_SHAPE
    assert fwd(rows_=-1) == E_SHAPE
    assert fwd(V_=96) == E_UNSUP
    assert fwd(V_=512) == E_UNSUP
    assert fwd(eps=-1.0) == E_SHAPE
    assert fwd(eps=float("nan")) == E_SHAPE
    assert fwd(z=None) == E_NULL
    assert fwd(w=None) == E_NULL
    assert fwd(y=P(FAKE + 8)) == E_ALIGN
    assert fwd(y=o) == E_ALIAS
    need = L.tla_out_gate_workspace_bytes(rows, V)
    assert need >= 128 * 4 and need % 256 == 0
    assert L.tla_out_gate_workspace_bytes(rows, 100) == 0
    ws = P(FAKE + 0x8000000)
    dy, do_, dz, dw = (P(FAKE + 0x4000000 + i * 0x1000000) for i in range(4))

    def bwd(ws_bytes=need, **kw):
        a = dict(dy=dy, do_=do_, dz=dz, dw=dw, ws=ws)
        a.update(kw)
        return L.tla_out_gate_bwd(tla.F32, rows, V, o, z, w, 1e-6, a["dy"], a["do_"], a["dz"], a["dw"],
                                  a["ws"], ws_bytes, None)
    assert bwd(ws_bytes=need - 1) == E_WS
    assert bwd(ws=None) == E_WS
    assert bwd(dw=None) == E_NULL
    assert bwd(dz=dy) == E_ALIAS
    assert bwd(dz=do_) == E_ALIAS


def test_gate_heads_validation():
    """Gate heads: dtype, shape, required and paired pointers, alignment,
    aliasing and workspace are checked on the host (fake addresses, nothing
    launched)."""
    L = tla.lib()
    P = ctypes.c_void_p
    x, xb, A, b, g, beta = (P(FAKE + i * 0x1000000) for i in range(6))
    n, H, E = 1000, 8, 8

    def fwd(dtype=tla.BF16, n_=n, H_=H, E_=E, **kw):
        a = dict(x=x, xb=xb, A=A, b=b, g=g, beta=beta)
        a.update(kw)
        return L.tla_gate_heads_fwd(dtype, n_, H_, E_, a["x"], a["xb"], a["A"], a["b"], a["g"], a["beta"],
                                    None)
    assert fwd(dtype=7) == E_SHAPE
    assert fwd(n_=-1) == E_SHAPE
    assert fwd(H_=0) == E_SHAPE
    assert fwd(E_=0) == E_SHAPE
    assert fwd(H_=2048, E_=1024) == E_SHAPE
    assert fwd(A=None) == E_NULL
    assert fwd(g=None) == E_NULL
    assert fwd(beta=None) == E_NULL      # xb without beta
    assert fwd(xb=None) == E_NULL        # beta without xb
    assert fwd(g=P(FAKE + 4)) == E_ALIGN
    assert fwd(g=x) == E_ALIAS
    assert fwd(beta=g) == E_ALIAS
    need = L.tla_gate_heads_workspace_bytes(n, H, E)
    assert need >= 2 * H * E * 4 and need % 256 == 0
    assert L.tla_gate_heads_workspace_bytes(n, 0, E) == 0
    dg, dbeta, dx, dxb, dA, db = (P(FAKE + 0x8000000 + i * 0x1000000) for i in range(6))
    ws = P(FAKE + 0x10000000)

    def bwd(ws_bytes=need, **kw):
        a = dict(xb=xb, dg=dg, dbeta=dbeta, dx=dx, dxb=dxb, dA=dA, db=db, ws=ws)
        a.update(kw)
        return L.tla_gate_heads_bwd(tla.F32, n, H, E, x, a["xb"], A, b, a["dg"], a["dbeta"], a["dx"],
                                    a["dxb"], a["dA"], a["db"], a["ws"], ws_bytes, None)
    assert bwd(ws_bytes=need - 1) == E_WS
    assert bwd(ws=None) == E_WS
    assert bwd(dA=None) == E_NULL
    assert bwd(dxb=None) == E_NULL
    assert bwd(dx=dg) == E_ALIAS
    assert bwd(db=dA) == E_ALIAS
    assert bwd(ws=dx) == E_ALIAS


def test_conv_in_validation():
    """Input side: dtype, widths, taps, group alignment, required pointers,
    alignment, aliasing and workspace are checked on the host (fake
    addresses, nothing launched)."""
    L = tla.lib()
    P = ctypes.c_void_p
    y, w, q, k, v, q2, k2 = (P(FAKE + i * 0x4000000) for i in range(7))
    shp = dict(B=2, T=100, H=8, K=128, V=128, E=8, W=4)

    def fwd(dtype=tla.BF16, eps=1e-6, **kw):
        a = dict(shp, y=y, w=w, q=q, k=k, v=v, q2=q2, k2=k2)
        a.update(kw)
        return L.tla_conv_in_fwd(dtype, a["B"], a["T"], a["H"], a["K"], a["V"], a["E"], a["W"], eps, a["y"],
                                 a["w"], a["q"], a["k"], a["v"], a["q2"], a["k2"], None)
    assert fwd(dtype=5) == E_SHAPE
    assert fwd(T=-1) == E_SHAPE
    assert fwd(H=0) == E_SHAPE
    assert fwd(K=96) == E_UNSUP
    assert fwd(E=4) == E_UNSUP
    assert fwd(V=12) == E_UNSUP
    assert fwd(W=5) == E_UNSUP
    assert fwd(W=0) == E_UNSUP
    assert fwd(H=1, K=8, V=8, E=16) == E_UNSUP  # q2 block would start inside a norm group
    assert fwd(eps=float("inf")) == E_SHAPE
    assert fwd(v=None) == E_NULL
    assert fwd(w=None) == E_NULL
    assert fwd(q=P(FAKE + 2)) == E_ALIGN
    assert fwd(k2=y) == E_ALIAS
    assert fwd(k=q) == E_ALIAS
    need = L.tla_conv_in_workspace_bytes(2, 100, 8, 128, 128, 8, 4)
    assert need > 0 and need % 256 == 0
    dq, dk, dv, dq2, dk2, dy, dw = (P(FAKE + 0x40000000 + i * 0x4000000) for i in range(7))
    ws = P(FAKE + 0x80000000)

    def bwd(ws_bytes=need, **kw):
        a = dict(dq=dq, dk=dk, dv=dv, dq2=dq2, dk2=dk2, dy=dy, dw=dw, ws=ws)
        a.update(kw)
        return L.tla_conv_in_bwd(tla.F32, 2, 100, 8, 128, 128, 8, 4, 1e-6, y, w, a["dq"], a["dk"], a["dv"],
                                 a["dq2"], a["dk2"], a["dy"], a["dw"], a["ws"], ws_bytes, None)
    assert bwd(ws_bytes=need - 1) == E_WS
    assert bwd(ws=None) == E_WS
    assert bwd(dw=None) == E_NULL
    assert bwd(dy=dq) == E_ALIAS
    assert bwd(dw=dy) == E_ALIAS


def test_proj_in_validation():
    """Fused input projection: widths, d_model, taps, group alignment,
    required pointers, alignment, aliasing and workspace are checked on the
    host (fake addresses, nothing launched)."""
    L = tla.lib()
    P = ctypes.c_void_p
    u, Wp, w, q, k, v, q2, k2, y = (P(FAKE + i * 0x4000000) for i in range(9))
    shp = dict(B=2, T=100, Dm=256, H=8, K=128, V=128, E=8, W=4)

    def fwd(eps=1e-6, **kw):
        a = dict(shp, u=u, Wp=Wp, w=w, q=q, k=k, v=v, q2=q2, k2=k2, y=y)
        a.update(kw)
        return L.tla_proj_in_fwd(a["B"], a["T"], a["Dm"], a["H"], a["K"], a["V"], a["E"], a["W"], eps,
                                 a["u"], a["Wp"], a["w"], a["q"], a["k"], a["v"], a["q2"], a["k2"],
                                 a["y"], None)
    assert fwd(T=-1) == E_SHAPE
    assert fwd(H=0) == E_SHAPE
    assert fwd(K=256) == E_UNSUP  # a channel tile holds whole heads (at most 128)
    assert fwd(E=4) == E_UNSUP
    assert fwd(Dm=12) == E_UNSUP
    assert fwd(Dm=0) == E_UNSUP
    assert fwd(W=5) == E_UNSUP
    assert fwd(H=1, K=8, V=8, E=16) == E_UNSUP
    assert fwd(eps=float("nan")) == E_SHAPE
    assert fwd(Wp=None) == E_NULL
    assert fwd(k2=None) == E_NULL
    assert fwd(q=P(FAKE + 8)) == E_ALIGN
    assert fwd(q=u) == E_ALIAS
    assert fwd(y=k) == E_ALIAS
    assert fwd(B=0, u=None, q=None, k=None, v=None, q2=None, k2=None, y=None) == 0  # nothing to do
    need = L.tla_proj_in_workspace_bytes(2, 100, 256, 8, 128, 128, 8, 4)
    assert need > 0 and need % 256 == 0
    dq, dk, dv, dq2, dk2, du, dWp, dw = (P(FAKE + 0x40000000 + i * 0x4000000) for i in range(8))
    ws = P(FAKE + 0x80000000)

    def bwd(ws_bytes=need, **kw):
        a = dict(dq=dq, dk=dk, dv=dv, dq2=dq2, dk2=dk2, du=du, dWp=dWp, dw=dw, ws=ws, y=y)
        a.update(kw)
        return L.tla_proj_in_bwd(2, 100, 256, 8, 128, 128, 8, 4, 1e-6, u, Wp, w, a["y"], a["dq"], a["dk"],
                                 a["dv"], a["dq2"], a["dk2"], a["du"], a["dWp"], a["dw"], a["ws"],
                                 ws_bytes, None)
    assert bwd(ws_bytes=need - 1) == E_WS
    assert bwd(ws=None) == E_WS
    assert bwd(y=None) == E_NULL
    assert bwd(dWp=None) == E_NULL
    assert bwd(du=dq) == E_ALIAS
    assert bwd(dWp=dw) == E_ALIAS


def test_mfma_rate_validation_and_flop_count():
    """The MFMA-rate diagnostic checks its arguments on the host; its FLOP
    count is 4 waves x rounds x (32 x 16x16x32 or 8 x 32x32x16) per block."""
    L = tla.lib()
    P = ctypes.c_void_p
    assert L.tla_mfma_rate(2, 256, 10, P(FAKE), None) == E_SHAPE
    assert L.tla_mfma_rate(0, 0, 10, P(FAKE), None) == E_SHAPE
    assert L.tla_mfma_rate(1, 256, 0, P(FAKE), None) == E_SHAPE
    assert L.tla_mfma_rate(0, 256, 10, None, None) == E_NULL
    assert L.tla_mfma_rate(0, 256, 10, P(FAKE + 4), None) == E_ALIGN
    assert L.tla_mfma_rate_flop(0, 256, 10) == 256 * 4 * 10 * 32 * 16 * 16 * 32 * 2
    assert L.tla_mfma_rate_flop(1, 256, 10) == 256 * 4 * 10 * 8 * 32 * 32 * 16 * 2
    assert L.tla_mfma_rate_flop(3, 256, 10) == 0


def test_noalloc_rejects_oversized_call_on_the_host():
    """tla_fwd_noalloc checks its scratch need before any HIP call."""
    L = tla.lib()
    desc = tla.make_desc(tla.GDN, 4, 4096, 8, 128, 128, 8, 64, tla.BF16, tla.BF16)
    nul = ctypes.c_void_p(None)
    assert L.tla_fwd_noalloc(ctypes.byref(desc), *([nul] * 10), nul) == E_WS
    assert b"scratch" in L.tla_last_error()
    bad = tla.make_desc(tla.GDN, 4, 4096, 8, 128, 128, 3, 64, tla.BF16, tla.BF16)
    assert L.tla_fwd_noalloc(ctypes.byref(bad), *([nul] * 10), nul) == E_UNSUP

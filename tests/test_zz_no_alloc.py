"""tla_fwd_noalloc (the inference forward on the library's static device
scratch) against tla_fwd with a caller workspace and against the fp64
oracle, through the C ABI: two calls in a row on one GPU, the second with a
smaller input (the scratch keeps the first call's contents), plus the
rejection of a call whose workspace need exceeds the scratch."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2609_36529_amd as tla
from paper_2609_36529_amd import synth
from helpers import TOL_BF16, TOL_F32, dev, host64, rel_err

pytestmark = pytest.mark.gpu
NAMES = ("q", "k", "v", "q2", "k2", "g")


def one(variant, dtype, B, T, H, E=8, seed=61):
    cfg = synth.Config("noalloc", variant, B, T, H, 128, 128, E, 64, dtype, "softplus16",
                       variant == tla.GDN, 0.02, seed)
    inp = synth.make_inputs(cfg)
    d = {k: dev(v) for k, v in inp.items()}
    args = [d[n] for n in NAMES] + [d["beta"], d["s0"]]
    o_na = torch.empty(d["v"].shape, dtype=torch.float32, device="cuda")
    sf_na = torch.empty((B, H, E, 128, 128), dtype=torch.float32, device="cuda")
    o_na, sf_na = tla.fwd_noalloc(variant, *args, chunk=64, out_dtype=torch.float32, o=o_na,
                                  s_final=sf_na)
    o_ws, sf_ws, _ = tla.fwd(variant, *args, chunk=64, out_dtype=torch.float32)
    torch.cuda.synchronize()
    # the same kernels on the same inputs: bitwise equal to the workspace call
    assert torch.equal(o_na, o_ws) and torch.equal(sf_na, sf_ws)
    ro, rs = oracle.fwd(variant, *[synth.to64(inp[n]) for n in NAMES], synth.to64(inp["beta"]),
                        synth.to64(inp["s0"]))
    tol = TOL_F32 if dtype == "f32" else TOL_BF16
    eo, es = rel_err(host64(o_na), ro), rel_err(host64(sf_na), rs)
    print(f"noalloc variant={variant} {dtype} B={B} T={T} H={H}: o err {eo:.2e} s_final err {es:.2e}",
          flush=True)
    assert eo <= tol and es <= tol, (eo, es)


@pytest.mark.parametrize("variant", [tla.SGLA, tla.GDN])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_two_calls_second_smaller(variant, dtype):
    one(variant, dtype, B=2, T=517, H=4, seed=61)
    one(variant, dtype, B=1, T=77, H=2, seed=62)


def test_noalloc_rejects_oversized_call_without_launch():
    L = tla.lib()
    # B4 H8 T4096 K = V = 128 E8 chunk 64: about 147 MB of per-chunk workspace
    desc = tla.make_desc(tla.GDN, 4, 4096, 8, 128, 128, 8, 64, tla.BF16, tla.BF16)
    assert tla.workspace_bytes(desc, tla.OP_FWD) > tla.NOALLOC_SCRATCH_BYTES
    nul = ctypes.c_void_p(None)
    rc = L.tla_fwd_noalloc(ctypes.byref(desc), *([nul] * 10), nul)
    assert rc == 5, rc  # TLA_E_WORKSPACE, before any pointer is used
    assert b"scratch" in L.tla_last_error()

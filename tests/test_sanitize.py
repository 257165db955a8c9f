"""Address and undefined-behaviour sanitizer builds of the host code, run on
the CPU: the fp64 oracle (oracle/tla_oracle.c, driven by
oracle/sanitize_check.c over both variants, optional beta / initial state /
final-state gradient, lengths across the backward's checkpoint segment, and
one decode step against the forward) and the C ABI's host-side validation
(tla_api.cpp with its host code instrumented, driven by
tests/sanitize/api_check.cpp with calls that are all rejected before any
device work, plus the size queries).  A sanitizer report fails the build's
run (-fno-sanitize-recover)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE = os.path.join(ROOT, "oracle")
CSRC = os.path.join(ROOT, "paper_2609_36529_amd", "csrc")
BUILD = os.path.join(ROOT, "paper_2609_36529_amd", "_build")
ROCM = "/opt/rocm"
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r


def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-std=c99", "-O1", "-g", "-fopenmp", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", "-Wall", "-Wextra", os.path.join(ORACLE, "tla_oracle.c"),
          os.path.join(ORACLE, "sanitize_check.c"), "-o", exe, "-lm"])
    r = _run([exe], env=dict(ENV, OMP_NUM_THREADS="4"), timeout=300)
    assert "sanitize check: ok" in r.stdout


@pytest.mark.skipif(not os.path.exists(os.path.join(ROCM, "bin", "hipcc")), reason="needs hipcc")
def test_abi_host_validation_under_asan_ubsan(tmp_path):
    objs = [os.path.join(BUILD, f + ".o") for f in
            ("tla_fwd.hip", "tla_bwd.hip", "tla_step.hip", "tla_gate.hip", "tla_conv.hip",
             "tla_proj.hip", "tla_diag.hip")]
    if not all(os.path.exists(o) for o in objs):
        from paper_2609_36529_amd import build as hip_build
        hip_build.build()
    api_o, chk_o, exe = (str(tmp_path / n) for n in ("api.o", "chk.o", "api_check"))
    # the device part of tla_api.cpp is built as usual; only its host code is instrumented
    _run([os.path.join(ROCM, "bin", "hipcc"), "-x", "hip", "--offload-arch=gfx950", "-std=c++17",
          "-O1", "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
          "-Xarch_host", "-fno-sanitize-recover=all", "-Xclang", "-target-feature", "-Xclang",
          "-packed-fp32-ops", "-c", os.path.join(CSRC, "tla_api.cpp"), "-o", api_o])
    cxx = os.path.join(ROCM, "llvm", "bin", "clang++")
    if not os.path.exists(cxx):
        cxx = shutil.which("clang++") or cxx
    _run([cxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-c", os.path.join(ROOT, "tests", "sanitize", "api_check.cpp"), "-o", chk_o])
    _run([cxx, "-fsanitize=address,undefined", chk_o, api_o, *objs, "-L" + os.path.join(ROCM, "lib"),
          "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", exe])
    r = _run([exe], env=dict(ENV, ASAN_OPTIONS="detect_leaks=0"), timeout=120)
    assert "api check: ok" in r.stdout

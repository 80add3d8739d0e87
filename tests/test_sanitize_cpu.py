"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds the C-ABI layer (csrc/api.cpp, host code only: its validation, dispatch
and workspace arithmetic) and the oracle (oracle/lb_oracle.c) with the host
sanitizers, links them with tests/sanitize/abi_driver.cpp against the built
library (for the kernels' host-side geometry functions) and runs the driver:
every validation path of the boundary, the pure helpers over extreme sizes, a
600-linear list, and the oracle's pack, unpack, forward (serial and OpenMP),
latent and dense routes on a small layer.  No GPU call is made."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2506_13771_amd")
LIB = os.path.join(PKG, "liblittlebit.so")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]


def _run(cmd, **kw):
    res = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert res.returncode == 0, f"{' '.join(cmd)}\n{res.stdout}\n{res.stderr}"
    return res


@pytest.mark.skipif(not os.path.exists(LIB) or not os.path.exists(HIPCC), reason="library or hipcc missing")
def test_abi_and_oracle_under_sanitizers(tmp_path):
    inc = os.path.join(ROOT, "include")
    common = ["-x", "hip", "--offload-host-only", "-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer", "-I", inc]
    # api.cpp holds a device array (the no-allocation entry point's scratch): its device side is
    # compiled too (no kernels, so it is quick), the sanitizers apply to the host side only
    full = ["-x", "hip", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-O1",
            "-g", "-std=c++17", "-fno-omit-frame-pointer", "-I", inc]
    api_o, drv_o, orc_o, exe = (str(tmp_path / n) for n in ("api.o", "driver.o", "oracle.o", "driver"))
    _run([HIPCC] + full + SAN + ["-c", os.path.join(PKG, "csrc", "api.cpp"), "-o", api_o])
    _run([HIPCC] + common + SAN + ["-c", os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp"), "-o", drv_o])
    _run(["gcc", "-c", "-O1", "-g", "-std=c99", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
          "-ffp-contract=off", "-fopenmp", os.path.join(ROOT, "oracle", "lb_oracle.c"), "-o", orc_o])
    _run([HIPCC] + SAN + ["--offload-arch=gfx950", "-fopenmp", drv_o, api_o, orc_o, "-L" + PKG, "-llittlebit",
                          "-Wl,-rpath," + PKG,
                          "-o", exe])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    res = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "sanitized host checks passed" in res.stdout
    assert "runtime error" not in res.stderr and "AddressSanitizer" not in res.stderr, res.stderr

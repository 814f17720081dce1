"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two drivers in tests/sanitize/ are built with the sanitizers and run:
  * oracle_driver.c with oracle/fibattn_oracle.c (gcc): every oracle entry point on
    small inputs that reach the edge cases of the attended set;
  * abi_driver.cpp with a host-sanitized build of the C ABI (api.hip; the kernels'
    objects are linked as built): every entry point on paths that return before any
    HIP call (rung tables, workspace sizes, refusals of invalid arguments).
Any invalid access, leak or undefined operation makes the driver exit non-zero.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
KERNEL_OBJS = ["fwd", "bwd", "rope", "fwd_mfma", "bwd_mfma", "alpha"]
# sanitizers on the host side only: each flag is handed to the host compilation
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout}\n{r.stderr}"
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-O1", "-g", "-std=c99", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
          "-fno-omit-frame-pointer", "-fopenmp", "-o", exe, os.path.join(SAN, "oracle_driver.c"),
          os.path.join(ROOT, "oracle", "fibattn_oracle.c"), "-lm"])
    r = _run([exe], env=ENV, timeout=300)
    assert r.stdout.strip().endswith("OK")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="needs hipcc")
def test_abi_host_code_under_sanitizers(tmp_path):
    objs = [os.path.join(ROOT, "_build", o + ".o") for o in KERNEL_OBJS]
    if not all(os.path.exists(o) for o in objs):
        from paper_2606_28560_amd.build import build
        build()
    api = str(tmp_path / "api_san.o")
    drv = str(tmp_path / "abi_driver.o")
    exe = str(tmp_path / "abi_san")
    inc = ["-I", os.path.join(ROOT, "include")]
    _run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-fPIC", "-std=c++17", "-Xclang", "-target-feature",
          "-Xclang", "-packed-fp32-ops", *inc, *HOST_SAN, "-c",
          os.path.join(ROOT, "paper_2606_28560_amd", "csrc", "api.hip"), "-o", api])
    _run([HIPCC, "-O1", "-g", "-std=c++17", *inc, *HOST_SAN, "-c", os.path.join(SAN, "abi_driver.cpp"),
          "-o", drv])
    _run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, "-o", exe, drv, api, *objs])
    r = _run([exe], env=ENV, timeout=300)
    assert r.stdout.strip().endswith("OK")

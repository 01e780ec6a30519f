"""AddressSanitizer / UndefinedBehaviorSanitizer builds of the host code (CPU only).

* The float64 oracle (oracle/mea_oracle.c) with a native driver that calls
  every entry point (tests/native/oracle_check.c), built with gcc.
* The C ABI's host code -- validation, planning, workspace carving in
  paper_2112_05682_amd/csrc/api.hip -- with the kernel launchers replaced by
  recording stubs (tests/native/launch_stubs.cpp) and a driver that checks the
  recorded plans (tests/native/abi_check.cpp).  api.hip is built for gfx950
  as in the library, with the sanitizers applied to its host side only
  (-Xarch_host); no kernel runs.

Any sanitizer report makes the driver exit non-zero (-fno-sanitize-recover).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    noise = "is not a recognized feature for this target"
    err = "\n".join(ln for ln in r.stderr.splitlines() if noise not in ln)
    assert r.returncode == 0, "%s\n%s\n%s" % (" ".join(cmd), r.stdout[-3000:], err[-3000:])
    return r.stdout


def test_oracle_under_address_and_undefined_sanitizers(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("needs gcc")
    exe = str(tmp_path / "oracle_check")
    _run(["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", "-fopenmp", "-Wall", "-Wextra", "-Werror",
          os.path.join(ROOT, "oracle", "mea_oracle.c"), os.path.join(NATIVE, "oracle_check.c"),
          "-o", exe, "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", OMP_NUM_THREADS="4")
    out = _run([exe], env=env, timeout=300)
    assert "oracle_check ok" in out


def test_c_abi_host_code_under_address_and_undefined_sanitizers(tmp_path):
    if not os.path.exists(HIPCC):
        pytest.skip("needs hipcc")
    inc = "-I" + os.path.join(ROOT, "include")
    common = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", *HOST_SAN, inc]
    api_o, stubs_o, drv_o = (str(tmp_path / n) for n in ("api.o", "stubs.o", "abi_check.o"))
    _run([HIPCC, "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          *common, "-c", os.path.join(ROOT, "paper_2112_05682_amd", "csrc", "api.hip"), "-o", api_o])
    for src, obj in (("launch_stubs.cpp", stubs_o), ("abi_check.cpp", drv_o)):
        _run([HIPCC, "--offload-host-only", "-x", "hip", *common, "-c", os.path.join(NATIVE, src),
              "-o", obj])
    exe = str(tmp_path / "abi_check")
    _run([HIPCC, "--offload-arch=gfx950", *HOST_SAN, api_o, stubs_o, drv_o, "-o", exe])
    # The HIP runtime's own start-up allocations are not this code's: leaks off.
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    out = _run([exe], env=env, timeout=300)
    assert "abi_check ok" in out

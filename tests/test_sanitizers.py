"""CPU code under AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

* The oracle: built with gcc -fsanitize=address,undefined (no recovery) and
  driven by the whole pin suite in a child Python process that preloads the
  ASan runtime.
* The library's host code (argument checks, workspace layouts, launch
  planning, the timing state): every source compiled as for the library,
  with ASan and UBSan on the host side only (the kernels are not
  instrumented), linked into a small C++ driver
  (tests/sanitize/abi_checks.cpp) that calls every entry point with rejected
  arguments and with empty batches, which run the whole validation and
  layout code and return before any launch.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
OUT = os.path.join(ROOT, "_build", "sanitize")
CSRC = os.path.join(ROOT, "paper_2607_26475_amd", "csrc")
SOURCES = ("ckv_kernels.hip", "ckv_api.cpp", "ckv_profile.cpp", "ckv_pipeline.cpp")
ENV_NO_LEAKS = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1",
                "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1"}


def _hipcc():
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    pytest.skip("hipcc not found")


def _run(cmd, env=None, timeout=600):
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-4000:]}\n{r.stderr[-4000:]}"
    return r


def test_oracle_pins_under_asan_ubsan():
    import oracle
    os.makedirs(OUT, exist_ok=True)
    lib = os.path.join(OUT, "libckv_oracle_asan.so")
    oracle.build(out=lib, extra=("-g", "-fno-omit-frame-pointer", "-fsanitize=address",
                                 "-fsanitize=undefined", "-fno-sanitize-recover=all"))
    runtime = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                             text=True, check=True).stdout.strip()
    assert os.path.exists(runtime), runtime
    env = dict(os.environ, CKV_ORACLE_LIB=lib, LD_PRELOAD=runtime, **ENV_NO_LEAKS)
    r = _run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
              os.path.join(HERE, "test_oracle.py")], env=env)
    assert " passed" in r.stdout and "failed" not in r.stdout, r.stdout[-2000:]


def test_host_code_under_asan_ubsan():
    hipcc = _hipcc()
    os.makedirs(OUT, exist_ok=True)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    common = ["-O1", "-g", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
              f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}"]
    objs = []
    for src in SOURCES:
        obj = os.path.join(OUT, src + ".asan.o")
        _run([hipcc, "-x", "hip", *common, *san, "-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    drv = os.path.join(OUT, "abi_checks.o")
    _run([hipcc, "-x", "hip", *common, *san, "-c",
          os.path.join(HERE, "sanitize", "abi_checks.cpp"), "-o", drv])
    exe = os.path.join(OUT, "abi_checks")
    _run([hipcc, "--offload-arch=gfx950", *san, *objs, drv, "-o", exe])
    r = _run([exe], env=dict(os.environ, **ENV_NO_LEAKS), timeout=300)
    assert "abi checks ok" in r.stdout

"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

1. The ABI layer (argument validation, workspace sizing, the exact partition
   arithmetic) is built with host-side sanitizers against launch stubs that
   abort, and tests/sanitize/abi_checks.cpp drives its error paths: every
   rejected call must return its status without reaching a launch.
2. Both C oracles are built with gcc's sanitizers and their pin tests run
   against that build (loaded through SF_ORACLE_LIB, the runtimes preloaded).
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_06838_amd", "csrc")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
SAN_ENV = {"ASAN_OPTIONS": "detect_leaks=0:verify_asan_link_order=0", "UBSAN_OPTIONS": "print_stacktrace=1"}


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_abi_validation_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_checks")
    # sanitizers on the host pass only (the device pass of this file holds no kernels)
    cmd = [HIPCC, "-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, os.path.join(CSRC, "sf_abi.hip"),
           os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "abi_checks.cpp"), "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120, env={**os.environ, **SAN_ENV})
    assert res.returncode == 0, res.stdout + res.stderr
    assert "abi checks passed" in res.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracles_under_sanitizers(tmp_path):
    lib = str(tmp_path / "liboracle_san.so")
    srcs = [os.path.join(ROOT, "oracle", f) for f in ("sf_oracle.c", "gdn_oracle.c")]
    subprocess.run(["gcc", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", *srcs, "-o", lib, "-lm"],
                   check=True, capture_output=True, text=True)
    rt = [subprocess.run(["gcc", f"-print-file-name={n}"], capture_output=True, text=True).stdout.strip()
          for n in ("libasan.so", "libubsan.so")]
    env = {**os.environ, **SAN_ENV, "SF_ORACLE_LIB": lib, "LD_PRELOAD": " ".join(rt)}
    # the sanitized build is the one mapped
    probe = subprocess.run([sys.executable, "-c", "import oracle; oracle._load(); print(open('/proc/self/maps').read())"],
                           cwd=ROOT, capture_output=True, text=True, env=env, timeout=300)
    assert probe.returncode == 0, probe.stderr[-2000:]
    assert lib in probe.stdout
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          "tests/test_oracle_pins.py", "tests/test_gdn_oracle_pins.py"],
                         cwd=ROOT, capture_output=True, text=True, env=env, timeout=900)
    assert res.returncode == 0, (res.stdout + res.stderr)[-4000:]
    assert "passed" in res.stdout

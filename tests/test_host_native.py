"""Host-side native checks, built with AddressSanitizer and UBSan (CPU only).

* The C ABI layer (``csrc/api.cpp``) linked with host stand-ins for the HIP
  runtime and the kernel launchers (``tests/native/abi_stubs.cpp``): every
  entry point runs through validation to its dispatch, and the resolved
  problem is checked (``tests/native/abi_driver.cpp``).
* The persistent block-indexer work split (``csrc/persistent_units.hpp``)
  replayed over many sequence lengths, first groups and grid sizes: every
  (query group, key tile) unit is covered exactly once.
* The oracle's C source built with both sanitizers and run under the oracle
  pin tests.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_07703_amd", "csrc")
NATIVE = os.path.join(ROOT, "tests", "native")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
HIP_HOST = ["-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]


def _gxx(out, srcs, extra=()):
    cmd = ["g++", "-std=c++17", "-O1", "-g", *SAN, *HIP_HOST, "-I", os.path.join(ROOT, "include"),
           "-I", CSRC, *srcs, "-o", out, *extra]
    subprocess.run(cmd, check=True, capture_output=True, text=True)


def _run(exe, env=None):
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    return r.stdout


def test_abi_layer_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_driver")
    _gxx(exe, [os.path.join(CSRC, "api.cpp"), os.path.join(NATIVE, "abi_stubs.cpp"),
               os.path.join(NATIVE, "abi_driver.cpp")])
    assert "abi ok" in _run(exe)


def test_persistent_split_covers_every_unit_once(tmp_path):
    exe = str(tmp_path / "unit_cover")
    _gxx(exe, [os.path.join(NATIVE, "unit_cover.cpp")])
    assert "cover ok" in _run(exe)


def _runtime(name):
    return subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True,
                          text=True, check=True).stdout.strip()


def test_oracle_pins_under_sanitizers(tmp_path):
    lib = str(tmp_path / "libsp_oracle_san.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c99", "-fopenmp", "-fPIC", "-shared", *SAN,
                    os.path.join(ROOT, "oracle", "sp_oracle.c"), "-o", lib, "-lm"],
                   check=True, capture_output=True, text=True)
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not (os.path.isabs(asan) and os.path.isabs(ubsan)):
        pytest.skip("sanitizer runtimes not found")
    env = dict(os.environ, SP_ORACLE_LIB=lib, LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    probe = ("import oracle; oracle._load(); import sys; "
             "sys.exit(0 if oracle._lib._name == sys.argv[1] else 3)")
    subprocess.run([sys.executable, "-c", probe, lib], check=True, env=env, cwd=ROOT,
                   timeout=120)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "tests/test_oracle_pins.py", "tests/test_oracle_next_pins.py"],
                       capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "passed" in r.stdout

"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two programs are built with gcc/g++ ``-fsanitize=address,undefined`` and run:

* ``sanitize/host_driver.cpp`` links the host side of the HIP library
  (``csrc/jfkv_host.cpp``: page allocator, argument validation, snapshot
  writer and reader) against CPU stand-ins for the HIP runtime calls and the
  kernel launchers (``sanitize/stubs.cpp``); the page-run copy runs on the
  CPU, so snapshot save and restore round-trip real bytes through files.
* ``sanitize/oracle_driver.c`` runs every entry point of the C oracle on
  small ragged inputs, invalid page IDs and rejected arguments.

No GPU code is built: only host sources, with the host compiler.  A finding
of either sanitizer ends its program with a non-zero status (recovery is
compiled out), which fails the test."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2609_17475_amd", "csrc")
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
       "-fno-sanitize-recover=all", "-static-libasan", "-static-libubsan"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None,
                                reason="host compilers not found")


def _run(cmd, **kw):
    p = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert p.returncode == 0, "%s\nrc=%d\n%s%s" % (" ".join(cmd), p.returncode, p.stdout,
                                                  p.stderr[-4000:])
    return p


def _env():
    env = dict(os.environ)
    env["ASAN_OPTIONS"] = "detect_leaks=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    return env


def _check_clean(p, banner):
    out = p.stdout + p.stderr
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert banner in p.stdout


def test_host_library_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_driver")
    _run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
          "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
          os.path.join(CSRC, "jfkv_host.cpp"), os.path.join(HERE, "stubs.cpp"),
          os.path.join(HERE, "host_driver.cpp"), "-o", exe])
    p = _run([exe], timeout=300, env=_env())
    _check_clean(p, "checks passed")


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-std=c11", *SAN, "-ffp-contract=off", "-fno-fast-math",
          "-I" + os.path.join(ROOT, "oracle"), os.path.join(ROOT, "oracle", "jf_oracle.c"),
          os.path.join(HERE, "oracle_driver.c"), "-o", exe, "-lm"])
    p = _run([exe], timeout=300, env=_env())
    _check_clean(p, "checks passed")

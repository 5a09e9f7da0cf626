"""Host-only AddressSanitizer / UndefinedBehaviorSanitizer runs (no GPU):
the C oracle and the library's host packers, each built with the sanitizers
from its own sources and driven over ragged shapes by a small program in
tests/sanitize/.  The GPU code of the packer's source is compiled without
them (the sanitizer flags apply to the host side only)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SAN = ["-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]


def _run(exe):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    env.pop("LD_PRELOAD", None)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ERROR" not in r.stderr and "runtime error" not in r.stderr, r.stderr


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    subprocess.run(["gcc", "-O1", "-g", "-std=c11", "-pthread", *SAN,
                    os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"),
                    os.path.join(ROOT, "oracle", "sherry_oracle.c"), "-o", exe, "-lm"],
                   check=True, capture_output=True, timeout=300)
    _run(exe)


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_host_packer_under_sanitizers(tmp_path):
    exe = str(tmp_path / "pack_driver")
    host_san = [f for flag in SAN for f in ("-Xarch_host", flag)]
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", *host_san,
                    "-I" + os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "paper_2601_07892_amd", "csrc", "pack.hip"),
                    os.path.join(ROOT, "tests", "sanitize", "pack_driver.cpp"), "-o", exe],
                   check=True, capture_output=True, timeout=600)
    _run(exe)

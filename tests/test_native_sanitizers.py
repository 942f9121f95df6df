"""Host builds of the C-ABI validation layer and of the oracle under
AddressSanitizer + UndefinedBehaviorSanitizer (g++/gcc only, no GPU code):
every entry point is driven through valid and invalid arguments, and every
oracle function runs on tiny arrays, with sanitizer errors fatal."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
NATIVE = os.path.join(ROOT, "tests", "native")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stdout + r.stderr
    return r.stdout


def test_abi_validation_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_driver")
    _run(["g++", "-std=c++17", *SAN, "-I", os.path.join(ROOT, "include"),
          "-I", os.path.join(ROOT, "paper_2607_21224_amd", "csrc"),
          os.path.join(ROOT, "paper_2607_21224_amd", "csrc", "cpdp_api.cpp"),
          os.path.join(NATIVE, "stub_launch.cpp"), os.path.join(NATIVE, "abi_driver.cpp"),
          "-o", exe])
    out = _run([exe], env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
    assert out.strip().startswith("OK"), out


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-std=c11", *SAN, "-ffp-contract=off",
          os.path.join(ROOT, "oracle", "cpdp_oracle.c"),
          os.path.join(NATIVE, "oracle_driver.c"), "-lm", "-o", exe])
    out = _run([exe], env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
    assert "oracle checksum" in out

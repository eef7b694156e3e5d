"""Sanitizer builds (CPU only): the C oracle and the host side of the C ABI,
compiled with AddressSanitizer and UndefinedBehaviorSanitizer and run over
every function and entry point (tests/sanitize/): the oracle on small inputs
with exactly-sized buffers and every edge case of n and N; the host side over
valid and invalid arguments of every call, its device launches replaced by
stubs that report no device, so that validation, the LDS and split plans and
the workspace layout all run."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g",
       "-O1"]
ROCM_INCLUDE = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, (" ".join(cmd), r.stdout[-2000:], r.stderr[-2000:])
    return r.stdout


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-std=c99", *SAN, "-o", exe, os.path.join(HERE, "sanitize", "oracle_main.c"),
          os.path.join(ROOT, "oracle", "vdref.c"), "-lm"])
    out = _run([exe], env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"}, timeout=300)
    assert "oracle sanitizer run ok" in out


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_abi_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_san")
    _run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I", ROCM_INCLUDE,
          "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2609_23314_amd", "csrc"),
          "-o", exe, os.path.join(HERE, "sanitize", "host_main.cpp"),
          os.path.join(ROOT, "paper_2609_23314_amd", "csrc", "vd_api.cpp")])
    out = _run([exe], env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1"}, timeout=300)
    assert "host sanitizer run ok" in out

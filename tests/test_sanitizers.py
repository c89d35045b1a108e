"""CPU-only runs under AddressSanitizer and UndefinedBehaviorSanitizer.

* the oracle (plain C) on small shapes, zero-padded widths and n_dyad above a
  width included, checked against the dense weight its own forward pass spans;
* the C-ABI layer (argument checks, pass descriptions, workspace checks) built
  host-only with mock kernel launchers, including a launcher that fails, which
  must come back as DYAD_ERR_LAUNCH.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CLANG = "/opt/rocm/llvm/bin/clang++"
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300, **kw)
    assert r.returncode == 0, f"{' '.join(cmd)}\n{r.stdout[-3000:]}\n{r.stderr[-3000:]}"
    return r


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_check")
    _run(["gcc", "-std=c11", "-fopenmp", *SAN, "-o", exe, os.path.join(HERE, "oracle_check.c"),
          os.path.join(ROOT, "oracle", "dyad_oracle.c"), "-lm"])
    r = _run([exe], env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1", "OMP_NUM_THREADS": "2"})
    assert "oracle sanitized ok" in r.stdout


@pytest.mark.skipif(not os.path.exists(CLANG), reason="ROCm clang not installed")
def test_abi_layer_under_sanitizers_with_mock_launchers(tmp_path):
    exe = str(tmp_path / "abi_mock")
    csrc = os.path.join(ROOT, "paper_2312_06881_amd", "csrc")
    # host-only build: no device code is compiled, the launchers are the mocks
    cmd = [CLANG, "-x", "hip", "--offload-host-only", "-std=c++17", *SAN,
           "-I", os.path.join(ROOT, "include"), "-I", csrc,
           os.path.join(csrc, "dyad_abi.hip"), os.path.join(HERE, "abi_mock.cpp"),
           "-o", exe, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"]
    _run(cmd)
    r = _run([exe], env={**os.environ, "ASAN_OPTIONS": "detect_leaks=0"})
    assert "abi mock ok" in r.stdout

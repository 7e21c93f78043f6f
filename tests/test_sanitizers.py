"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the host code (CPU only).

* The C oracle with tests/sanitize/oracle_main.c: every entry point on small
  shapes (rectangular, post-padded, batch-padded with lengths 0, 1 and whole
  blocks of padding, the objective, exact attention) and its argument
  checks, OpenMP on, leak checking on.
* The C ABI's host code (monarch_attn.hip, sanitizers on its host pass) with
  tests/sanitize/abi_main.cpp, which stands in for the dispatch units: the
  argument checks of every entry point, the shape queries and workspace
  sizes, head counts at and beyond the grid limit, and the empty calls.  No
  call reaches a HIP function.

Any report of either sanitizer fails the run (-fno-sanitize-recover=all).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
HIPCC = "/opt/rocm/bin/hipcc"


def _run(cmd, env=None, timeout=300):
    res = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=timeout)
    assert res.returncode == 0, (cmd, res.stdout[-4000:], res.stderr[-4000:])
    return res.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_san")
    _run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fsanitize=address,undefined",
          "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
          os.path.join(ROOT, "oracle", "monarch_oracle.c"), os.path.join(SAN, "oracle_main.c"), "-o", exe, "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", OMP_NUM_THREADS="4")
    assert "ok" in _run([exe], env=env)


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_abi_host_code_under_asan_ubsan(tmp_path):
    # every sanitizer flag applies to the host pass only (the device pass holds
    # only the scratch array of the no-allocation entry point)
    common = [HIPCC, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
              "-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
              "-fno-omit-frame-pointer", '-DMA_BUILD_ID="0123456789abcdef"', "-I", os.path.join(ROOT, "include")]
    abi_o, main_o, exe = (str(tmp_path / x) for x in ("abi.o", "main.o", "abi_san"))
    _run(common + ["-c", os.path.join(ROOT, "paper_2505_18698_amd", "csrc", "monarch_attn.hip"), "-o", abi_o])
    _run(common + ["--cuda-host-only", "-x", "hip", "-c", os.path.join(SAN, "abi_main.cpp"), "-o", main_o])
    _run([HIPCC, "--offload-arch=gfx950", "-Xarch_host", "-fsanitize=address,undefined", abi_o, main_o, "-o", exe])
    # the HIP runtime keeps allocations of its own to the end of the process: no leak check here
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    assert "ok" in _run([exe], env=env)

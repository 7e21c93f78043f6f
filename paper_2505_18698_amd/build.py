"""Build the HIP library libmonarch_attn.so in-tree for gfx950 with hipcc.

Each translation unit of csrc/ (the C ABI and one dispatch unit per element
type) is compiled separately and in parallel, then linked into one shared
library.
"""
from __future__ import annotations

import concurrent.futures
import glob
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libmonarch_attn.so")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # Packed-FP32 VALU forms are disabled; the compiler emits scalar fp32 ops instead.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def sources() -> list[str]:
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


HEADER = os.path.join(ROOT, "include", "monarch_attn.h")


def source_hash() -> str:
    """First 16 hex digits of a SHA-256 over every file the library is built
    from (csrc/*.hip, csrc/*.hpp and the C header), names and contents, in
    name order.  Compiled into the library as monarch_attn_build_id(); the
    binding compares the two at import."""
    import hashlib

    h = hashlib.sha256()
    files = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.hpp"))) + [HEADER]
    for path in files:
        h.update(os.path.relpath(path, ROOT).encode())
        h.update(b"\0")
        with open(path, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    return h.hexdigest()[:16]


def _run(cmd):
    res = subprocess.run(cmd, capture_output=True, text=True)
    return res.returncode, res.stdout + res.stderr


def build(verbose: bool = False, extra_flags=()) -> str:
    cc = hipcc()
    build_id = f'-DMA_BUILD_ID="{source_hash()}"'
    with tempfile.TemporaryDirectory(prefix="ma_build_") as tmp:
        objs, jobs = [], []
        for src in sources():
            obj = os.path.join(tmp, os.path.basename(src) + ".o")
            objs.append(obj)
            jobs.append([cc, *FLAGS, build_id, *extra_flags, "-I", os.path.join(ROOT, "include"), "-c", src, "-o", obj])
        workers = min(len(jobs), max(1, min(8, os.cpu_count() or 1)))
        with concurrent.futures.ThreadPoolExecutor(workers) as ex:
            results = list(ex.map(_run, jobs))
        for (rc, log), job in zip(results, jobs):
            if rc != 0:
                sys.stderr.write(log)
                raise RuntimeError(f"hipcc failed on {job[-3]}")
            if verbose:
                sys.stderr.write(log)
        tmp_lib = LIB + ".tmp"
        rc, log = _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp_lib])
        if rc != 0:
            sys.stderr.write(log)
            raise RuntimeError("linking libmonarch_attn.so failed")
        os.replace(tmp_lib, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))

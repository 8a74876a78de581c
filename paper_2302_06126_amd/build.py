"""Compile the HIP sources into the in-tree C-ABI library ``libtag.so`` (gfx950).

Each source file is compiled to an object in parallel (one hipcc per file),
then the objects are linked into the shared library.  Every call compiles
every file."""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "libtag.so")

# hipcc flags: gfx950 only; packed-fp32 code generation is switched off (the
# host pass warns that it does not know the feature, which is harmless).
ARCH = ["--offload-arch=gfx950"]
CFLAGS = ["-O3", "-std=c++17", "-fPIC",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-mllvm", "-amdgpu-mfma-vgpr-form",
          "-Wno-unused-result", "-I" + os.path.join(ROOT, "include")]


def sources():
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def _hipcc() -> str:
    return shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def _run(cmd) -> tuple:
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines() if "packed-fp32-ops" not in l)
    return res.returncode, out


def build(verbose: bool = False, jobs: int = 0) -> str:
    hipcc = _hipcc()
    srcs = sources()
    jobs = jobs or max(1, min(len(srcs), os.cpu_count() or 1, 16))
    with tempfile.TemporaryDirectory(prefix="tag_build_") as tmpd:
        objs = [os.path.join(tmpd, os.path.basename(s) + ".o") for s in srcs]
        cmds = [[hipcc, *ARCH, *CFLAGS, "-c", s, "-o", o] for s, o in zip(srcs, objs)]
        if verbose:
            for c in cmds:
                print(" ".join(c), flush=True)
        with ThreadPoolExecutor(max_workers=jobs) as ex:
            results = list(ex.map(_run, cmds))
        failed = False
        for (rc, out), s in zip(results, srcs):
            if rc != 0:
                failed = True
                sys.stderr.write(f"--- {os.path.basename(s)}\n{out}\n")
            elif verbose and out.strip():
                print(out)
        if failed:
            raise RuntimeError("hipcc failed")
        tmp = LIB + ".tmp"
        link = [hipcc, *ARCH, "-shared", "-fPIC", *objs, "-o", tmp]
        if verbose:
            print(" ".join(link), flush=True)
        rc, out = _run(link)
        if rc != 0:
            sys.stderr.write(out + "\n")
            raise RuntimeError("hipcc link failed")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)

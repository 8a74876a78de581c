"""CPU sanitizer builds of the library's host code and of the oracle.

AddressSanitizer + UndefinedBehaviorSanitizer ("address"), or
ThreadSanitizer ("thread"), for running the CPU tests of the host search,
the host simulator (and its thread pool) and the oracle under them
(tests/test_sanitize.py).  Only the host pass of each HIP source is
instrumented; device code is compiled as usual.  The outputs are separate
libraries (libtag_asan.so / libtag_tsan.so next to libtag.so, and
oracle/liboracle_asan.so / liboracle_tsan.so), loaded through the
TAG_LIBRARY and TAG_ORACLE_LIBRARY environment variables with the matching
clang runtime preloaded (runtime_path)."""
from __future__ import annotations

import glob
import os
import subprocess
import tempfile
from concurrent.futures import ThreadPoolExecutor

from . import build as B

LLVM = "/opt/rocm/llvm"

# host-pass flags, every sanitizer option directly after -Xarch_host
HOST_FLAGS = {
    "address": ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-shared-libsan",
                "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"],
    "thread": ["-Xarch_host", "-fsanitize=thread", "-Xarch_host", "-shared-libsan",
               "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-g"],
}
ORACLE_FLAGS = {
    "address": ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-shared-libsan"],
    "thread": ["-fsanitize=thread", "-shared-libsan"],
}
SUFFIX = {"address": "asan", "thread": "tsan"}


def runtime_path(kind: str) -> str:
    """The clang sanitizer runtime to preload for `kind`."""
    name = {"address": "libclang_rt.asan-x86_64.so", "thread": "libclang_rt.tsan-x86_64.so"}[kind]
    hits = sorted(glob.glob(os.path.join(LLVM, "lib", "clang", "*", "lib", "linux", name)))
    if not hits:
        raise RuntimeError(f"{name} not found under {LLVM}")
    return hits[-1]


def build_library(kind: str, verbose: bool = False) -> str:
    """libtag_<asan|tsan>.so from the same sources as libtag.so."""
    hipcc = B._hipcc()
    out = os.path.join(B.HERE, f"libtag_{SUFFIX[kind]}.so")
    srcs = B.sources()
    with tempfile.TemporaryDirectory(prefix="tag_san_") as tmpd:
        objs = [os.path.join(tmpd, os.path.basename(s) + ".o") for s in srcs]
        cmds = [[hipcc, *B.ARCH, *B.CFLAGS, *HOST_FLAGS[kind], "-c", s, "-o", o] for s, o in zip(srcs, objs)]
        with ThreadPoolExecutor(max_workers=max(1, min(len(srcs), os.cpu_count() or 1, 16))) as ex:
            results = list(ex.map(B._run, cmds))
        for (rc, log), s in zip(results, srcs):
            if rc != 0:
                raise RuntimeError(f"hipcc failed on {os.path.basename(s)}:\n{log}")
            if verbose and log.strip():
                print(log)
        rc, log = B._run([hipcc, *B.ARCH, "-shared", "-fPIC", *HOST_FLAGS[kind], *objs, "-o", out])
        if rc != 0:
            raise RuntimeError(f"link failed:\n{log}")
    return out


def build_oracle(kind: str) -> str:
    """oracle/liboracle_<asan|tsan>.so (plain C99, instrumented)."""
    src = os.path.join(B.ROOT, "oracle", "tag_oracle.c")
    out = os.path.join(B.ROOT, "oracle", f"liboracle_{SUFFIX[kind]}.so")
    subprocess.check_call([os.path.join(LLVM, "bin", "clang"), "-O1", "-g", "-std=c99", "-fPIC", "-shared",
                           "-fno-omit-frame-pointer", *ORACLE_FLAGS[kind], "-o", out, src, "-lm"])
    return out


def environment(kind: str, lib: str, oracle_lib: str) -> dict:
    """Environment of a process that runs the CPU tests on the sanitized libraries."""
    env = dict(os.environ)
    env["LD_PRELOAD"] = runtime_path(kind)
    env["TAG_LIBRARY"] = lib
    env["TAG_ORACLE_LIBRARY"] = oracle_lib
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["TSAN_OPTIONS"] = "halt_on_error=1:report_signal_unsafe=0"
    return env

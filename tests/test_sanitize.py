"""The CPU tests of the host search, the host simulator and the oracle,
rerun in a child process on sanitizer builds of the library's host code and
of the oracle: AddressSanitizer + UndefinedBehaviorSanitizer, and
ThreadSanitizer (the simulator's and the state packer's host thread pools).
The builds take minutes, so the test runs only with TAG_SANITIZE=1:

    TAG_SANITIZE=1 python -m pytest tests/test_sanitize.py -q
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(os.environ.get("TAG_SANITIZE") != "1",
                                reason="sanitizer builds run with TAG_SANITIZE=1")

TESTS = {"address": ["tests/test_search.py", "tests/test_simulate.py", "tests/test_sim_oracle.py",
                     "tests/test_oracle_pins.py", "tests/test_abi.py"],
         "thread": ["tests/test_simulate.py", "tests/test_search.py"]}


@pytest.mark.parametrize("kind", ["address", "thread"])
def test_cpu_suites_under_sanitizer(kind):
    sys.path.insert(0, ROOT)
    from paper_2302_06126_amd import sanitize as S
    lib = S.build_library(kind)
    olib = S.build_oracle(kind)
    env = S.environment(kind, lib, olib)
    # the builds carry the instrumentation, and the child loads them
    probe = {"address": "__asan_report", "thread": "__tsan_"}[kind]
    for path in (lib, olib):
        syms = subprocess.run(["nm", "-D", path], stdout=subprocess.PIPE, text=True).stdout
        assert probe in syms, path
    chk = subprocess.run([sys.executable, "-c", "import oracle, paper_2302_06126_amd._abi as a; a.load(); "
                          "oracle.lib(); print(a.LIB_PATH)"], cwd=ROOT, env=env, stdout=subprocess.PIPE,
                         stderr=subprocess.STDOUT, text=True, timeout=600)
    assert chk.returncode == 0 and chk.stdout.strip().endswith(os.path.basename(lib)), chk.stdout[-2000:]
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu", *TESTS[kind]]
    res = subprocess.run(cmd, cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                         timeout=3000)
    out = res.stdout
    print(out[-3000:])
    for marker in ("ERROR: AddressSanitizer", "runtime error:", "WARNING: ThreadSanitizer", "ERROR: ThreadSanitizer"):
        assert marker not in out, marker
    assert res.returncode == 0

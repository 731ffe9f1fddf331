"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

Every library source is compiled with the sanitizers on its host code only
(the device code is built as usual) and linked with tests/abi_host_check.cpp,
a driver that calls every entry point that needs no GPU with valid arguments,
each documented error case and boundary values (validation, workspace sizes,
energy split, calls without a context, context creation on a device that
does not exist).  The run must report no sanitizer finding (UB aborts:
-fno-sanitize-recover) and no failed expectation.
"""
import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _build():
    from paper_2609_36692_amd import _build as B
    if not os.path.exists(B.HIPCC):
        pytest.skip("hipcc not available")
    out = os.path.join(B.OBJ_DIR, "san")
    os.makedirs(out, exist_ok=True)
    # Host-only sanitizers: each -fsanitize= right after -Xarch_host.
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
           "-Xarch_host", "-g"]
    srcs = [os.path.join(B.CSRC, s) for s in B.SOURCES] + [os.path.join(ROOT, "tests", "abi_host_check.cpp")]

    def compile_one(path):
        obj = os.path.join(out, os.path.splitext(os.path.basename(path))[0] + ".o")
        cmd = [B.HIPCC, *B.COMMON, *san, "-c", path, "-o", obj]
        if path.endswith(".cpp"):
            cmd[1:1] = ["-x", "hip"]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
        return obj

    with ThreadPoolExecutor(max_workers=min(len(srcs), int(os.environ.get("MAX_JOBS", "4")) or 1)) as ex:
        objs = list(ex.map(compile_one, srcs))
    exe = os.path.join(out, "abi_host_check")
    r = subprocess.run([B.HIPCC, f"--offload-arch={B.ARCH}", *san, "-o", exe, *objs], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def test_host_abi_under_asan_and_ubsan():
    exe = _build()
    env = dict(os.environ, ASAN_OPTIONS="halt_on_error=1:detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    log = r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in log and "runtime error" not in log, log
    assert "ERROR: LeakSanitizer" not in log, log
    assert r.returncode == 0 and "0 failure(s)" in r.stdout, log

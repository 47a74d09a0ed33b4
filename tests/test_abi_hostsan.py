"""The C ABI's host-side argument checks under AddressSanitizer and
UndefinedBehaviorSanitizer: sn_api.cpp is built with g++ and both
sanitizers (the kernels are the regular objects) and tests/test_abi_cpu.py
runs against that library in a child process with the ASan runtime
preloaded.  Any sanitizer report aborts the child and fails this test."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    gxx = shutil.which("g++")
    if not gxx:
        return None
    r = subprocess.run([gxx, "-print-file-name=libasan.so"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_abi_checks_under_asan_and_ubsan():
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("g++ with the ASan runtime is not available")
    from paper_2506_01260_amd import build as b
    lib = b.build_host_sanitized()
    env = dict(os.environ)
    env.update(SN_LIBRARY=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    # the child loads the instrumented library with the ASan runtime in place
    probe = ("import paper_2506_01260_amd as sn; sn.lib(); "
             "maps = open('/proc/self/maps').read(); "
             "print(sn.LIB_PATH, 'libasan' in maps, 'libsn_hostsan' in maps)")
    r = subprocess.run([sys.executable, "-c", probe], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0 and r.stdout.split()[-2:] == ["True", "True"], r.stdout + r.stderr
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert " passed" in r.stdout

"""The host side of the C ABI under AddressSanitizer and UndefinedBehaviorSanitizer: runtime.hip
(shape, mask, workspace, argument and status checks, layouts, the host closure and signatures)
is rebuilt with both sanitizers on its host code, and the CPU ABI tests run against that build
in a child process with the sanitizer runtime preloaded; any report fails the run. No GPU is
needed: every call the tests make is rejected or answered on the host."""
import os
import subprocess
import sys

import pytest

from paper_2609_29499_amd import build as BLD

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(900)
def test_abi_host_checks_clean_under_asan_and_ubsan(tmp_path):
    if not os.path.exists(BLD.HIPCC):
        pytest.skip("hipcc is not available")
    lib = BLD.build_sanitized(str(tmp_path))
    rt = BLD.asan_runtime()
    assert os.path.exists(rt), rt
    pre = os.environ.get("LD_PRELOAD", "")
    env = dict(os.environ, TASP_LIB=lib, LD_PRELOAD=rt + (":" + pre if pre else ""),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    # the child loads the sanitized build, not the regular one
    probe = ("from paper_2609_29499_amd import binding as B; B.load(); "
             "m = open('/proc/self/maps').read(); "
             "print(B.LIB_PATH, 'libtasp_san.so' in m, 'asan' in m)")
    r = subprocess.run([sys.executable, "-c", probe], env=env, cwd=ROOT, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-3000:]
    assert r.stdout.split() == [lib, "True", "True"], r.stdout
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       env=env, cwd=ROOT, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0 and "passed" in r.stdout, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]

"""The host layer under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The library is rebuilt with both sanitizers on its host code (build.py --sanitize: every
-fsanitize= goes through -Xarch_host, device code is unchanged) and the C-ABI tests run
against it in a child process with the ASan runtime preloaded: argument validation,
workspace sizing and carving, the fault-injection path.  Any sanitizer report aborts the
child and fails this test with the report.  (It found an out-of-range enum load in
rp_create's dtype check.)
"""
import glob
import os
import subprocess
import sys

import pytest

from paper_2608_14498_amd import build as rbuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def _stale(lib):
    if not os.path.exists(lib):
        return True
    t = os.path.getmtime(lib)
    srcs = glob.glob(os.path.join(rbuild.CSRC, "*")) + [os.path.join(ROOT, "include", "rollplex.h")]
    return any(os.path.getmtime(s) > t for s in srcs)


def test_abi_tests_pass_under_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if rt is None or not os.path.exists(rbuild.HIPCC):
        pytest.skip("no hipcc or clang ASan runtime in this image")
    if _stale(rbuild.ASAN_LIB):
        rbuild.build(sanitize=True)
    log = str(tmp_path / "san")
    env = dict(os.environ, RP_LIBRARY=rbuild.ASAN_LIB, LD_PRELOAD=rt,
               ASAN_OPTIONS=f"detect_leaks=0:abort_on_error=1:log_path={log}",
               UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:log_path={log}")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi_cpu.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    reports = "".join(open(p).read() for p in glob.glob(log + "*"))
    assert r.returncode == 0 and not reports, (r.stdout[-3000:] + r.stderr[-3000:] + reports[:6000])
    assert "passed" in r.stdout

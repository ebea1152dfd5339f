"""The C-ABI layer under AddressSanitizer and UndefinedBehaviorSanitizer.

api.cpp (argument checks, overlap and span arithmetic, plans, workspace
layouts, error strings) is compiled by g++ with -fsanitize=address,undefined
and linked with the normal device objects; the CPU test files of the ABI and
the binding then run against that library in a child process with libasan
preloaded.  Any sanitizer report aborts the child and fails this test.  No
kernel is launched (there is no GPU here): kernels are not instrumented.
"""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_cpu_tests_under_host_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None or shutil.which("g++") is None:
        pytest.skip("g++ not available")
    libasan = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True,
                             text=True).stdout.strip()
    if not os.path.isabs(libasan) or not os.path.exists(libasan):
        pytest.skip("libasan not available")
    sys.path.insert(0, ROOT)
    from paper_2606_11660_amd import build as B
    try:
        lib = B.build_host_sanitized(str(tmp_path / "libattr_hostsan.so"))
    except RuntimeError as e:
        if "device objects missing" in str(e):
            pytest.skip(str(e))
        raise
    env = dict(os.environ)
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = libasan + (":" + pre if pre else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["ATTR_LIBRARY"] = lib
    # the child really loads the sanitized library
    probe = subprocess.run(
        [sys.executable, "-c",
         "import paper_2606_11660_amd as P; L = P.lib(); "
         "print(P.lib_path()); print(open('/proc/self/maps').read().count('libattr_hostsan'))"],
        cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert probe.returncode == 0, probe.stdout + probe.stderr
    path, n_maps = probe.stdout.split()[-2:]
    assert path == lib and int(n_maps) > 0
    r = subprocess.run(
        [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
         os.path.join(ROOT, "tests", "test_abi_cpu.py"),
         os.path.join(ROOT, "tests", "test_binding_cpu.py")],
        cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-4000:]
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr

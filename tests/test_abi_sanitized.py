"""The C interface's host code under AddressSanitizer and UBSan: the library
is rebuilt with the sanitizers on its host code only (device code is
unchanged) and the argument-checking tests of test_abi.py run against it in
a child process (no GPU needed)."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from paper_2405_19261_amd import build as lib_build  # noqa: E402


def test_abi_checks_under_host_asan_ubsan(tmp_path):
    rt = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not rt:
        pytest.skip("clang's AddressSanitizer runtime not found")
    out = str(tmp_path / "libspeccascade.so")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    lib_build.build(out=out, extra=san)
    env = dict(os.environ)
    env["SPC_LIB_PATH"] = out
    # the sanitizer runtime must come first among the preloaded libraries
    env["LD_PRELOAD"] = ":".join(x for x in (rt[-1], os.environ.get("LD_PRELOAD", "")) if x)
    env["ASAN_OPTIONS"] = "detect_leaks=0:exitcode=23"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       env=env, capture_output=True, text=True, timeout=900, cwd=ROOT)
    report = r.stdout[-3000:] + r.stderr[-3000:]
    assert r.returncode == 0, report
    assert "AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, report

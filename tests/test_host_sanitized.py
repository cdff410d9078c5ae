"""The host planner (layout.cpp, api.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer, CPU only: it is built with g++ against the
checking stub launchers of tests/sanitize/stub_launchers.cpp, and the host
test suite (random layouts per mask preset, every argument error) plus the
stub cases (random layouts through every entry and split choice) run against
it in a child process.  Any sanitizer report or broken schedule fails."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_21229_amd", "csrc")


def _runtime(name):
    out = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return out if os.path.isabs(out) and os.path.exists(out) else None


@pytest.mark.timeout(600)
def test_planner_clean_under_asan_ubsan(tmp_path):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("g++ has no AddressSanitizer runtime")
    lib = str(tmp_path / "librefcache_san.so")
    build = ["g++", "-std=c++17", "-O1", "-g", "-fPIC", "-shared", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"),
             "-I", CSRC, os.path.join(CSRC, "layout.cpp"), os.path.join(CSRC, "api.cpp"),
             os.path.join(ROOT, "tests", "sanitize", "stub_launchers.cpp"), "-o", lib]
    r = subprocess.run(build, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ)
    env["REFCACHE_LIB"] = lib
    env["REFCACHE_STUB"] = "1"
    # the ASan runtime must come first among the preloaded libraries
    env["LD_PRELOAD"] = ":".join(x for x in (asan, os.environ.get("LD_PRELOAD", "")) if x)
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    cmd = [sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
           os.path.join(ROOT, "tests", "test_capi_host.py"), os.path.join(ROOT, "tests", "sanitize", "stub_cases.py")]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in r.stdout and "skipped" not in r.stdout.split("\n")[-2], out[-2000:]

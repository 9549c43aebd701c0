"""AddressSanitizer and UndefinedBehaviorSanitizer over the host code: the
CPU oracle (every entry point, tests/sanitize/oracle_check.c) and the GPU
library's host-side table construction and conflict model
(tests/sanitize/host_tables_check.cpp over csrc/tables.cpp). Built with gcc /
g++ (host code only), run as child processes; any sanitizer report aborts the
child."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
       "-fno-sanitize-recover=all"]


def build_and_run(cmd, exe, tmp_path):
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    # verify_asan_link_order=0: the environment may preload a library ahead
    # of the sanitizer runtime; that is left as it is
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env,
                       cwd=str(tmp_path))
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ok" in r.stdout and "runtime error" not in r.stderr, r.stderr
    return r.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_sanitizers(tmp_path):
    o = os.path.join(ROOT, "oracle")
    exe = str(tmp_path / "oracle_check")
    srcs = [os.path.join(ROOT, "tests", "sanitize", "oracle_check.c")] + [
        os.path.join(o, f) for f in ("philox.c", "tables.c", "sampling.c", "sgns.c")]
    build_and_run(["gcc", *SAN, "-I" + o, *srcs, "-lm", "-o", exe], exe, tmp_path)


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not found")
def test_host_tables_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_check")
    csrc = os.path.join(ROOT, "paper_1611_06172_amd", "csrc")
    build_and_run(["g++", *SAN, "-std=c++17", "-I" + os.path.join(ROOT, "include"),
                   "-I" + csrc, os.path.join(ROOT, "tests", "sanitize", "host_tables_check.cpp"),
                   os.path.join(csrc, "tables.cpp"), "-o", exe], exe, tmp_path)

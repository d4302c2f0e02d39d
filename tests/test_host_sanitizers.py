"""The host libraries (page tags, scheduler, progress tracker) under
AddressSanitizer and UndefinedBehaviorSanitizer: tests/native/host_stress.cpp
drives them through their C ABI with random call sequences and checks the
invariants that hold for any sequence; any sanitizer report fails the test.
Built with g++ (host code only), run as its own process."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCES = [os.path.join(ROOT, "tests", "native", "host_stress.cpp")] + [
    os.path.join(ROOT, "paper_2606_17787_amd", "csrc", f)
    for f in ("lumen_page_tags.cpp", "lumen_sched.cpp", "lumen_progress.cpp")]


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_libraries_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "host_stress")
    build = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
             "-static-libasan", "-static-libubsan",
             "-I", os.path.join(ROOT, "include"), *SOURCES, "-o", exe]
    r = subprocess.run(build, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, "300"], capture_output=True, text=True,
                       timeout=300, env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "host stress ok: 300 rounds" in r.stdout

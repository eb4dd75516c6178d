"""Host-side logic of libpcs without a GPU, under AddressSanitizer and
UndefinedBehaviorSanitizer: the arena sub-allocator against a brute-force
occupancy model, plan descriptors against the ring's defining index map
(logical row t of ring o at physical row (head + t) mod capacity) and the
validation of bad descriptors, and the snapshot image header (round trips,
single-field corruptions, a size crafted to wrap 64-bit arithmetic, random
mutations and truncations).  The checks live in tests/host/test_host_logic.cpp,
which compiles the library's own host header (csrc/pcs_host.h) with g++."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "host", "test_host_logic.cpp")


def test_host_logic_under_sanitizers(tmp_path):
    cxx = shutil.which("g++")
    if cxx is None:
        pytest.skip("g++ is not installed")
    exe = str(tmp_path / "host_logic")
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-Wall", "-Wextra", "-Werror",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), SRC, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok "), r.stdout

"""The oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer.

The oracle is what every parity claim is measured against, so its C part
(oracle/pcs_oracle.c) is built a second time with both sanitizers and the
oracle's own pin tests are run against that build in a child interpreter
(sanitizer runtimes preloaded; leak checking off, as the interpreter itself
keeps memory until exit).  Any out-of-bounds access, use after free or
undefined arithmetic in the oracle fails the test."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["tests/test_oracle_hash.py", "tests/test_oracle_ring_classify.py", "tests/test_oracle_contract.py",
        "tests/test_oracle_image.py", "tests/test_oracle_bank.py", "tests/test_oracle_discover.py"]

PLUGIN = """
import oracle
oracle.build = lambda force=False: {lib!r}


def pytest_sessionfinish(session, exitstatus):
    print("\\noracle library:", oracle._L()._name)
"""


def _runtime(name):
    p = subprocess.run(["gcc", "-print-file-name=" + name], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


def test_oracle_pins_under_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc is not installed")
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("sanitizer runtimes are not installed")
    lib = str(tmp_path / "liboracle_sanitized.so")
    subprocess.run(["gcc", "-O1", "-g", "-std=c99", "-Wall", "-Wextra", "-Werror", "-fPIC", "-shared",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                    "-o", lib, os.path.join(ROOT, "oracle", "pcs_oracle.c")], check=True)
    (tmp_path / "sanitized_oracle.py").write_text(PLUGIN.format(lib=lib))
    env = dict(os.environ)
    env["LD_PRELOAD"] = ":".join([asan, ubsan] + ([env["LD_PRELOAD"]] if env.get("LD_PRELOAD") else []))
    env["ASAN_OPTIONS"] = "detect_leaks=0:verify_asan_link_order=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1"
    env["PYTHONPATH"] = os.pathsep.join([str(tmp_path), ROOT])
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "sanitized_oracle", "-p", "no:cacheprovider",
                        "-m", "not gpu", *PINS], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, (r.stdout[-3000:], r.stderr[-3000:])
    assert " passed" in r.stdout
    assert "oracle library: " + lib in r.stdout, r.stdout[-1000:]

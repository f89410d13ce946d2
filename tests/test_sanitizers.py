"""The oracle and the library's host code under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only): both are rebuilt with
-fsanitize=address,undefined (any finding aborts), and the CPU pins of the
oracle and the host entry points run against those builds in a child
process with the ASan runtime preloaded."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1911_13214_amd", "csrc")
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-shared", "-fPIC"]


def _runtime(name):
    p = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return p if os.path.isabs(p) and os.path.exists(p) else None


@pytest.fixture(scope="module")
def sanitized(tmp_path_factory):
    if not shutil.which("gcc") or not shutil.which("g++") or not _runtime("libasan.so"):
        pytest.skip("gcc with the ASan runtime is not available")
    d = tmp_path_factory.mktemp("san")
    oracle_so, host_so = str(d / "liboracle_san.so"), str(d / "librotor_host_san.so")
    subprocess.check_call(["gcc", "-std=c11", *SAN, os.path.join(ROOT, "oracle", "rotor_oracle.c"), "-o", oracle_so])
    subprocess.check_call(["g++", "-std=c++17", *SAN, "-fvisibility=hidden", "-I", os.path.join(ROOT, "include"),
                           "-I", CSRC, os.path.join(CSRC, "rotor_host.cpp"), os.path.join(CSRC, "rotor_plan.cpp"),
                           "-o", host_so])
    return oracle_so, host_so


def test_oracle_and_host_code_are_clean_under_asan_and_ubsan(sanitized):
    oracle_so, host_so = sanitized
    env = dict(os.environ, ROTOR_ORACLE_LIB=oracle_so, ROTOR_LIB=host_so, LD_PRELOAD=_runtime("libasan.so"),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               PYTHONDONTWRITEBYTECODE="1")
    # every CPU test of the oracle and of the host entry points, except
    # those about the full library's export table and its device entry points
    cmd = [sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-m", "not gpu",
           "tests/test_oracle_pins.py", "tests/test_frontend.py", "tests/test_abi.py", "tests/test_chaingen.py",
           "-k", "not exports_every and not hidden and not before_any_device_work"]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, tail

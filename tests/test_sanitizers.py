"""The host-only C / C++ code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU):
the oracle (oracle/pulse_oracle.c) and the admission search (csrc/ioaa.cpp) are built with
-fsanitize=address,undefined, and their tests (test_oracle_pins.py, test_ioaa.py) run against
those builds in a child process with the sanitizer runtimes preloaded.  Any report (an
out-of-bounds access, a use after free, undefined arithmetic) fails the child."""
import os
import subprocess
import sys

from oracle import build as obuild

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True,
                          check=True).stdout.strip()
    assert os.path.isabs(path) and os.path.exists(path), f"{name} not found"
    return path


def test_oracle_and_admission_search_under_asan_ubsan(tmp_path):
    oracle_lib = obuild.build_oracle_sanitized(str(tmp_path / "liboracle_asan.so"))
    ioaa_lib = str(tmp_path / "libioaa_asan.so")
    subprocess.run(["g++", "-O1", "-g", "-std=c++17", "-fPIC", "-shared", "-Wall", "-fno-omit-frame-pointer",
                    "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                    "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "paper_2609_34555_amd", "csrc", "ioaa.cpp"), "-o", ioaa_lib], check=True)
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": f"{_runtime('libasan.so')}:{_runtime('libubsan.so')}",
        "ASAN_OPTIONS": "detect_leaks=0:halt_on_error=1:verify_asan_link_order=0",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "PULSE_ORACLE_LIB": oracle_lib,
        "PULSE_SANITIZED_IOAA_LIB": ioaa_lib,
    })
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                          "tests/test_oracle_pins.py", "tests/test_ioaa.py"],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = res.stdout[-4000:] + res.stderr[-4000:]
    assert res.returncode == 0, out
    assert "AddressSanitizer" not in res.stderr and "runtime error" not in res.stderr, out
    assert " passed" in res.stdout and " failed" not in res.stdout, out

"""Build the CPU oracle (test infrastructure) into oracle/liboracle.so with gcc.

Plain -O2, strict IEEE semantics (no -ffast-math), single-threaded.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "pulse_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")


def build_oracle(verbose: bool = False) -> str:
    tmp = LIB + ".tmp"
    cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


def build_oracle_sanitized(out_path: str, verbose: bool = False) -> str:
    """The same source with AddressSanitizer and UndefinedBehaviorSanitizer (CPU only), for a
    test run of the pins under the sanitizers; load it with PULSE_ORACLE_LIB=out_path and the
    sanitizer runtimes preloaded."""
    cmd = ["gcc", "-O1", "-g", "-std=c99", "-fPIC", "-shared", "-Wall", "-Wextra", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-o", out_path, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return out_path


if __name__ == "__main__":
    print(build_oracle(verbose=True))

"""Build the C test program tests/c/abi_parity (plain C against include/pulse.h, linked with
libpulse.so, the oracle's liboracle.so and the HIP runtime), in place.  Test infrastructure."""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_parity.c")
EXE = os.path.join(HERE, "abi_parity")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build_c_tests(verbose: bool = False) -> str:
    tmp = EXE + ".tmp"
    cmd = ["gcc", "-std=c11", "-O1", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"), SRC, "-o", tmp,
           "-L", os.path.join(ROOT, "paper_2609_34555_amd"), "-lpulse", "-L", os.path.join(ROOT, "oracle"), "-loracle",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../paper_2609_34555_amd:$ORIGIN/../../oracle:" + os.path.join(ROCM, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build_c_tests(verbose=True))

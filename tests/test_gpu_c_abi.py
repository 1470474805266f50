"""The C ABI from plain C: tests/c/abi_parity runs one decode layer-step through libpulse.so
(pulse_build_digests, pulse_decode_layer) with no Python or torch in the process, and checks
every stage against the oracle (linked as a C library): digests bit-exact, selection up to
near-ties, table / free head / statistics / pool bytes exact, attention within 2e-3."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


def test_c_program_layer_step_matches_oracle():
    exe = os.path.join(HERE, "c", "abi_parity")
    print(f"\n[gpu] {exe}", flush=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    print(res.stdout + res.stderr, flush=True)
    assert res.returncode == 0, res.stderr
    assert "c abi parity ok" in res.stdout

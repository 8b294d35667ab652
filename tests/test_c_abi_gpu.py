"""The C ABI from plain C: tests/c_abi_parity.c verifies seeded batches with
asd_verify through the HIP runtime API alone (no C++, no Python binding) and
compares every output with the C oracle bit for bit.  __graft_entry__.build()
compiles it; it runs here as a child process."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

DRIVER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi_parity")


def test_pure_c_consumer_matches_the_oracle():
    assert os.path.exists(DRIVER), "tests/c_abi_parity is not built: run __graft_entry__.build()"
    print("case c_abi_parity: 40 seeded batches through asd_verify from C", flush=True)
    r = subprocess.run([DRIVER, "40"], capture_output=True, text=True, timeout=240)
    print(r.stdout[-3000:])
    assert r.returncode == 0, "exit %d\n%s\n%s" % (r.returncode, r.stdout[-2000:], r.stderr[-2000:])
    assert "40 of 40 cases matched the oracle" in r.stdout

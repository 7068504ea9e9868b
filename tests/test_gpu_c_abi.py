"""The boundary used from plain C: tests/c_abi_client.c, built by the package
build next to libc3.so, allocates with the HIP runtime and calls
c3_signature, c3_consensus and c3_localize with no Python or torch in the
process.  It checks clean replicas, one planted NaN and argument errors, and
prints "ok"."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT = os.path.join(ROOT, "paper_2608_11034_amd", "c3_abi_client")


def test_c_client_signature_consensus_localize():
    print("CASE c abi client", flush=True)
    assert os.path.exists(CLIENT), "c3_abi_client is not built: run __graft_entry__.build()"
    r = subprocess.run([CLIENT], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "ok"

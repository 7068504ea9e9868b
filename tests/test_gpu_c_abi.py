"""The boundary used from plain C: tests/c_abi_client.c, compiled here with
gcc (C99, no HIP compiler) against include/c3.h and linked to libc3.so,
allocates with the HIP runtime and calls c3_signature, c3_consensus and
c3_localize with no Python or torch in the process.  It checks clean
replicas, one planted NaN, a 130-replica vote and argument errors, and
prints "ok"."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.dirname(os.path.abspath(__file__))
LIBDIR = os.path.join(ROOT, "paper_2608_11034_amd")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    assert os.path.exists(os.path.join(LIBDIR, "libc3.so")), \
        "libc3.so is not built: run __graft_entry__.build()"
    exe = str(tmp_path_factory.mktemp("c_abi") / "c3_abi_client")
    cmd = [os.environ.get("CC", "gcc"), "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"),
           "-I", os.path.join(ROOT, "include"), os.path.join(HERE, "c_abi_client.c"), "-o", exe,
           "-L", LIBDIR, "-lc3", "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath," + LIBDIR, "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def test_c_client_signature_consensus_localize(client):
    print("CASE c abi client", flush=True)
    r = subprocess.run([client], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "ok"

"""The C ABI from plain C, with no Python in the path: tests/c_abi/closed_forms
(built by __graft_entry__.build(), linked to the in-tree libsdattn.so) runs
sdattn_forward on HIP-runtime buffers through every attention kernel and
checks the results Eq. 3 fixes in closed form (constant keys give the mean of
V, one key gives its value row bit for bit, a dominant key gives its row) and
that refused arguments leave the output untouched.  It runs as a child
process of the test session."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "closed_forms")


def test_c_client_closed_forms():
    if not os.path.exists(EXE):
        pytest.fail("tests/c_abi/closed_forms is not built (run __graft_entry__.build())")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(r.stdout)
    if r.returncode == 2:
        pytest.skip("no GPU visible to the C client")
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip().endswith("all cases ok"), r.stdout

"""The C ABI used from C++ with no Python in the process: tests/c_abi/epl_c_check allocates its own
device buffers, runs layout -> dispatch -> combine through include/epl.h on its own HIP stream (as
epl_layout + epl_dispatch, as one epl_layout_dispatch call and as its two phases), with packed rows
and with rows a pitch apart, plus the one-launch layer synchronised by Token-Flag Fusion and by
Data-for-Checksum, compares every output with the CPU oracle, and checks the documented error
statuses."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "epl_c_check")


def test_c_abi_standalone_program():
    if not os.path.exists(BIN):
        pytest.fail("tests/c_abi/epl_c_check is not built; run __graft_entry__.build()")
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=300)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c abi check ok" in r.stdout
    assert r.stdout.count(": ok") == 26  # 8 cases x 3 ways of calling, and the two layer variants

"""The library driven from plain C (tests/c_abi/abi_check.c): hipMalloc'd memory, its own
hipStream_t, the C ABI only.  The program compares five layers and two stacks fused across
depth with the oracle, checks that sequences run as segments with the state handoff equal
the single call bit for bit, and checks argument errors; it exits 0 when everything
matches."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu


def test_c_client_matches_oracle():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import c_abi
    if not os.path.exists(c_abi.BIN):
        c_abi.build()
    r = subprocess.run([c_abi.BIN], capture_output=True, text=True, timeout=300)
    print(r.stdout, r.stderr, flush=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "all cases match the oracle" in r.stdout

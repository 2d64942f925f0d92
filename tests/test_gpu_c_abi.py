"""GPU test: libattn.so called from C++ with the HIP runtime alone.

tests/c_abi/abi_check (built by __graft_entry__.build()) allocates its own
device buffers, runs attn_fwd and attn_decode on inputs with closed-form
results (identical V rows give that row; Q = 0 gives the mean of the allowed V
rows, full and causal; decode with Q = 0 and several split counts gives the
mean of V), and checks an unsupported head dimension is refused with a
message.  No Python or torch runs in that process, so this also shows the
library needs nothing from them.
"""
import os
import subprocess

import pytest

from tests.gpu_common import announce

pytestmark = pytest.mark.gpu

BIN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "abi_check")


def test_c_abi_caller_without_python():
    if not os.path.exists(BIN):
        pytest.fail("tests/c_abi/abi_check is not built: run __graft_entry__.build()")
    announce("tests/c_abi/abi_check (prefill and decode closed forms through the C ABI)")
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi_check ok" in r.stdout, r.stdout

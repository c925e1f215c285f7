"""The library used from plain C, through its C ABI alone: tests/c/abi_consumer
(built by ``__graft_entry__.build()``) allocates device memory with the HIP
runtime, runs an int32 bare scan and an fp32 fused scan whose results have
closed forms, and checks the rejection of a NULL output and of a host
pointer."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "c", "abi_consumer")


def test_plain_c_consumer():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(EXE), "tests/c/abi_consumer is missing: run __graft_entry__.build()"
    print("case: plain C consumer", flush=True)
    res = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "abi consumer ok" in res.stdout

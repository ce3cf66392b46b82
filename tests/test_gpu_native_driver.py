"""The C ABI from native code, no Python binding and no torch: tests/native/step_driver.cpp runs
two training steps of one table (the calls one by one through the multi-kernel coalesce, then
emb_train_step through the one-workgroup coalesce) and checks each against the CPU oracle
(lookup bit-exact, send layout bit-exact, sums within the fp32 summation bound, the update on its
own scale, rows not sent unchanged).  Built by __graft_entry__.build()."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

DRIVER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "native", "step_driver")


def test_native_driver_two_steps():
    assert os.path.exists(DRIVER), "tests/native/step_driver is missing: run __graft_entry__.build() first"
    r = subprocess.run([DRIVER], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "native driver: ok" in r.stdout, r.stdout
    assert "step 1:" in r.stdout and "step 2:" in r.stdout

"""The step executor's cross-stream order, checked on the host: step.hip is linked against stand-ins
that record every launch, signal write and wait, and event record and wait per stream, and a model of
the device runs the recorded work (tests/host_order/order_sim.cpp).  It must never wait for a value
that no write enqueued before it supplies, never let a signal word decrease, and never deadlock:
across handles reused between modes, a call that fails part-way, and a long random mix of modes and
single-stream schedules.  With a vector clock per stream it also checks happens-before: every two
launches that touch the same buffer of a set, or overlapping table rows, one of them writing, run in
the order the executor enqueued them, for every mode, events, signals and events under graph capture
(every stage's end an event record of its own, none attached to a dispatch), two to six buffer sets
with more steps than sets, and stream choices that include a set's streams changing between its uses;
and the two-thread enqueue (emb_train_step_queued: the library's worker thread enqueues each step's
lookup and update), each scenario several times so that the threads meet in different interleavings,
the steps' launches tagged from their arguments.  No GPU is used."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not found")
def test_step_signals_order_model(tmp_path):
    exe = tmp_path / "order_sim"
    cmd = [HIPCC, "-O1", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
           "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I",
           os.path.join(ROOT, "paper_2110_09132_amd", "csrc"), os.path.join(ROOT, "tests", "host_order", "order_sim.cpp"),
           "-x", "hip", os.path.join(ROOT, "paper_2110_09132_amd", "csrc", "step.hip"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, cwd=str(tmp_path))
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    lines = r.stdout.splitlines()
    assert lines[0].startswith("happens-before:") and lines[-1].startswith("ok:"), r.stdout
    assert any(l.startswith("queued:") for l in lines), r.stdout
